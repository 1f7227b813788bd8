// Rotary position embedding of query/key rows, in place: the post-RoPE Q and K that the
// scoring reads (App. "Draft-guided eviction implementation": queries recomputed post-RoPE
// from each layer's input; the compensation-token appendix: rotate-half pairs (i, i + d/2);
// Table "Backbones": theta = 500,000).  Pair i < d/2 of a row at position p turns by
// p * theta^(-2i/d).  The angle and the rotation are formed in double (positions reach
// 32K and more, where a float angle would be off by ~1e-3 rad) and rounded once to the
// stored type.  Elementwise and HBM-bound: one thread per (row, pair), consecutive
// threads on consecutive pairs of a row, looping over the heads.
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
  int64_t total;                // n_rows * half
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
  // one thread per (row, pair): the angle depends on those alone, so one sincos serves
  // the pair in every head
  for (int64_t t = (int64_t)blockIdx.x * kRopeThreads + threadIdx.x; t < a.total;
       t += (int64_t)gridDim.x * kRopeThreads) {
    const int i = (int)(t % a.half);
    const int r = (int)(t / a.half);
    double s, c;
    sincos((double)a.pos[r] * a.inv_freq[i], &s, &c);
    char* row = a.x + (int64_t)r * (2 * a.half) * a.elt;
    for (int h = 0; h < a.n_heads; ++h, row += a.head_stride_bytes) {
      if (a.elt == 2) {
        uint16_t* e = reinterpret_cast<uint16_t*>(row);
        const double x0 = bf16_to_f32(e[i]), x1 = bf16_to_f32(e[i + a.half]);
        e[i] = f32_to_bf16_rne((float)(x0 * c - x1 * s));
        e[i + a.half] = f32_to_bf16_rne((float)(x1 * c + x0 * s));
      } else {
        float* e = reinterpret_cast<float*>(row);
        const double x0 = e[i], x1 = e[i + a.half];
        e[i] = (float)(x0 * c - x1 * s);
        e[i + a.half] = (float)(x1 * c + x0 * s);
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
  a.total = (int64_t)n_rows * a.half;
  for (int i = 0; i < a.half; ++i) a.inv_freq[i] = pow(theta, -2.0 * i / head_dim);
  if (a.total == 0) return hipSuccess;
  const int64_t blocks = (a.total + kRopeThreads - 1) / kRopeThreads;
  const int grid = (int)(blocks < 65536 ? blocks : 65536);
  hipLaunchKernelGGL(rope_kernel, dim3(grid), dim3(kRopeThreads), 0, st, a);
  return hipGetLastError();
}

}  // namespace dge
