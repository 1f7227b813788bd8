// Rotary position embedding of query/key rows, in place: the post-RoPE Q and K that the
// scoring reads (App. "Draft-guided eviction implementation": queries recomputed post-RoPE
// from each layer's input; the compensation-token appendix: rotate-half pairs (i, i + d/2);
// Table "Backbones": theta = 500,000).  Pair i < d/2 of a row at position p turns by
// p * theta^(-2i/d).  The angle and the rotation are formed in double (positions reach
// 32K and more, where a float angle would be off by ~1e-3 rad) and rounded once to the
// stored type.  Elementwise and HBM-bound: one thread per (row, two neighbouring pairs),
// consecutive threads on consecutive pairs of a row, looping over the heads.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int kRopeThreads = 256;
constexpr int kMaxHalf = 64;   // head_dim <= 128

struct RopeArgs {
  char* x;
  const int32_t* pos;
  int64_t head_stride_bytes;
  int64_t total;                // n_rows * half / 2 (threads: two pairs each)
  int n_heads, n_rows, half, elt;
  double inv_freq[kMaxHalf];    // theta^(-2i/d), computed on the host
};

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }
__device__ __forceinline__ uint16_t f32_to_bf16_rne(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__global__ __launch_bounds__(kRopeThreads) void rope_kernel(RopeArgs a) {
  // one thread per (row, two neighbouring pairs i, i+1): the angles depend on those alone,
  // so their sines and cosines serve the pairs in every head; the two neighbours make the
  // accesses 4-byte (bf16) or 8-byte (float) wide
  const int pairs2 = a.half / 2;
  for (int64_t t = (int64_t)blockIdx.x * kRopeThreads + threadIdx.x; t < a.total;
       t += (int64_t)gridDim.x * kRopeThreads) {
    const int i = 2 * (int)(t % pairs2);
    const int r = (int)(t / pairs2);
    const double p = (double)a.pos[r];
    double s0, c0, s1, c1;
    sincos(p * a.inv_freq[i], &s0, &c0);
    sincos(p * a.inv_freq[i + 1], &s1, &c1);
    char* row = a.x + (int64_t)r * (2 * a.half) * a.elt;
    for (int h = 0; h < a.n_heads; ++h, row += a.head_stride_bytes) {
      if (a.elt == 2) {
        uint32_t* lo = reinterpret_cast<uint32_t*>(row + i * 2);
        uint32_t* hi = reinterpret_cast<uint32_t*>(row + (i + a.half) * 2);
        const uint32_t wl = *lo, wh = *hi;
        const double a0 = bf16_to_f32((uint16_t)(wl & 0xffffu)), a1 = bf16_to_f32((uint16_t)(wl >> 16));
        const double b0 = bf16_to_f32((uint16_t)(wh & 0xffffu)), b1 = bf16_to_f32((uint16_t)(wh >> 16));
        *lo = (uint32_t)f32_to_bf16_rne((float)(a0 * c0 - b0 * s0)) |
              ((uint32_t)f32_to_bf16_rne((float)(a1 * c1 - b1 * s1)) << 16);
        *hi = (uint32_t)f32_to_bf16_rne((float)(b0 * c0 + a0 * s0)) |
              ((uint32_t)f32_to_bf16_rne((float)(b1 * c1 + a1 * s1)) << 16);
      } else {
        float2* lo = reinterpret_cast<float2*>(row + i * 4);
        float2* hi = reinterpret_cast<float2*>(row + (i + a.half) * 4);
        const float2 va = *lo, vb = *hi;
        *lo = make_float2((float)((double)va.x * c0 - (double)vb.x * s0),
                          (float)((double)va.y * c1 - (double)vb.y * s1));
        *hi = make_float2((float)((double)vb.x * c0 + (double)va.x * s0),
                          (float)((double)vb.y * c1 + (double)va.y * s1));
      }
    }
  }
}

}  // namespace

hipError_t launch_rope(int n_heads, int n_rows, int head_dim, int dtype, int64_t head_stride,
                       const int32_t* positions, double theta, void* x, hipStream_t st) {
  RopeArgs a{};
  a.x = static_cast<char*>(x);
  a.pos = positions;
  a.elt = dtype == DGE_BF16 ? 2 : 4;
  a.head_stride_bytes = head_stride * a.elt;
  a.n_heads = n_heads;
  a.n_rows = n_rows;
  a.half = head_dim / 2;
  a.total = (int64_t)n_rows * (a.half / 2);
  for (int i = 0; i < a.half; ++i) a.inv_freq[i] = pow(theta, -2.0 * i / head_dim);
  if (a.total == 0) return hipSuccess;
  const int64_t blocks = (a.total + kRopeThreads - 1) / kRopeThreads;
  const int grid = (int)(blocks < 65536 ? blocks : 65536);
  hipLaunchKernelGGL(rope_kernel, dim3(grid), dim3(kRopeThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace dge
