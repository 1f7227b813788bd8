// Cache compaction (Alg. 1 step C; App. "Draft-guided eviction implementation", implementation notes):
//   out[b][h] = [ K[idx[b][h][0..n_kept)] , K[C_b .. N_b) , zero rows up to n_select + n_tail ]
// and the same for V.  Rows are copied as raw bytes, so the result is bit-exact for
// any element type.  Each thread moves one 16-byte piece of one row of K and the
// same piece of V; a row of head_dim elements is RB / 16 consecutive threads, so
// every wavefront reads and writes whole, contiguous rows.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

struct CompactArgs {
  const int32_t* idx;
  const int32_t* n_kept;
  const char* k;
  const char* v;
  char* k_out;
  char* v_out;
  SeqOffsets offs;
  int64_t head_stride_bytes;
  int n_kv_heads, n_select, n_tail, n_out;
};

template <int RB>
__global__ __launch_bounds__(256) void compact_kernel(CompactArgs a) {
  constexpr int TPR = RB / 16;            // threads per row
  constexpr int RPB = 256 / TPR;          // rows per block
  const int h = blockIdx.y, b = blockIdx.z;
  const int r = blockIdx.x * RPB + threadIdx.x / TPR;
  const int part = threadIdx.x % TPR;
  if (r >= a.n_out) return;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int C = N - a.n_tail;
  int nk = a.n_kept[b];
  nk = max(0, min(nk, min(a.n_select, C)));
  int src;
  if (r < nk) {
    src = a.idx[((int64_t)b * a.n_kv_heads + h) * a.n_select + r];
    src = max(0, min(src, C - 1));    // a malformed index never reads out of the sequence
  } else if (r < nk + a.n_tail) {
    src = C + (r - nk);
  } else {
    src = -1;
  }
  const int64_t o = (((int64_t)b * a.n_kv_heads + h) * a.n_out + r) * RB + part * 16;
  uint4 kv = make_uint4(0, 0, 0, 0), vv = make_uint4(0, 0, 0, 0);
  if (src >= 0) {
    const int64_t in = h * a.head_stride_bytes + (s0 + src) * RB + part * 16;
    kv = load16(a.k + in);
    vv = load16(a.v + in);
  }
  *reinterpret_cast<uint4*>(a.k_out + o) = kv;
  *reinterpret_cast<uint4*>(a.v_out + o) = vv;
}

template <int RB>
hipError_t launch_rb(const CompactArgs& a, const dge_geom_t& g, hipStream_t st) {
  constexpr int RPB = 256 / (RB / 16);
  dim3 grid((a.n_out + RPB - 1) / RPB, g.n_kv_heads, g.batch);
  hipLaunchKernelGGL((compact_kernel<RB>), grid, dim3(256), 0, st, a);
  return hipGetLastError();
}

// In-place compaction: the compacted rows of (b, h) overwrite the first n_kept + n_tail
// rows of that head's own segment of the cache.  Every retained row moves down or stays
// (idx is ascending, so idx[r] >= r; tail row t moves from C + t to n_kept + t).  One
// workgroup per (KV head, sequence) walks the output rows in chunks: it reads every
// source row of a chunk, meets a barrier, then writes the chunk.  The rows a chunk
// writes lie below every source of the later chunks (a source is never below its own
// output row), and the sources of this and the earlier chunks were read before the
// barrier, so no row is overwritten before it has been read.
constexpr int kInplaceThreads = 1024;
constexpr int kInplaceUnroll = 8;

template <int RB>
__global__ __launch_bounds__(kInplaceThreads) void compact_inplace_kernel(CompactArgs a,
                                                                         char* k, char* v) {
  constexpr int TPR = RB / 16;                    // threads per row
  constexpr int RPP = kInplaceThreads / TPR;      // rows per pass
  constexpr int CHUNK = RPP * kInplaceUnroll;     // rows read before each barrier
  const int h = blockIdx.x, b = blockIdx.y;
  const int sub = threadIdx.x / TPR, part = threadIdx.x % TPR;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int C = N - a.n_tail;
  const int nk = max(0, min(a.n_kept[b], min(a.n_select, C)));
  const int n_out = nk + a.n_tail;
  const int32_t* ix = a.idx + ((int64_t)b * a.n_kv_heads + h) * a.n_select;
  const int64_t base = h * a.head_stride_bytes + s0 * RB + part * 16;
  for (int c0 = 0; c0 < n_out; c0 += CHUNK) {
    uint4 kv[kInplaceUnroll], vv[kInplaceUnroll];
    int src[kInplaceUnroll];
#pragma unroll
    for (int u = 0; u < kInplaceUnroll; ++u) {
      const int r = c0 + u * RPP + sub;
      int s = -1;
      if (r < nk)
        s = max(r, min(ix[r], C - 1));   // a malformed index never moves a row upwards
      else if (r < n_out)
        s = C + (r - nk);
      src[u] = s == r ? -1 : s;          // a row already in place is not copied
      if (src[u] >= 0) {
        kv[u] = load16(k + base + (int64_t)src[u] * RB);
        vv[u] = load16(v + base + (int64_t)src[u] * RB);
      }
    }
    __syncthreads();   // every source row of this chunk has been read
#pragma unroll
    for (int u = 0; u < kInplaceUnroll; ++u) {
      if (src[u] >= 0) {
        const int r = c0 + u * RPP + sub;
        *reinterpret_cast<uint4*>(k + base + (int64_t)r * RB) = kv[u];
        *reinterpret_cast<uint4*>(v + base + (int64_t)r * RB) = vv[u];
      }
    }
  }
}

}  // namespace

hipError_t launch_compact_inplace(const dge_geom_t& g, const int32_t* idx, const int32_t* n_kept,
                                  int n_select, int n_tail, void* k, void* v, hipStream_t st) {
  CompactArgs a{};
  const int elt = g.dtype == DGE_BF16 ? 2 : 4;
  const int rb = g.head_dim * elt;
  a.idx = idx;
  a.n_kept = n_kept;
  a.offs = seq_offsets(g);
  a.head_stride_bytes = g.kv_head_stride * elt;
  a.n_kv_heads = g.n_kv_heads;
  a.n_select = n_select;
  a.n_tail = n_tail;
  a.n_out = n_select + n_tail;
  char* kc = static_cast<char*>(k);
  char* vc = static_cast<char*>(v);
  const dim3 grid(g.n_kv_heads, g.batch);
  switch (rb) {
    case 128: hipLaunchKernelGGL((compact_inplace_kernel<128>), grid, dim3(kInplaceThreads), 0, st, a, kc, vc); break;
    case 256: hipLaunchKernelGGL((compact_inplace_kernel<256>), grid, dim3(kInplaceThreads), 0, st, a, kc, vc); break;
    case 512: hipLaunchKernelGGL((compact_inplace_kernel<512>), grid, dim3(kInplaceThreads), 0, st, a, kc, vc); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_compact(const dge_geom_t& g, const int32_t* idx, const int32_t* n_kept,
                          int n_select, int n_tail, const void* k, const void* v, void* k_out,
                          void* v_out, hipStream_t st) {
  CompactArgs a{};
  const int elt = g.dtype == DGE_BF16 ? 2 : 4;
  const int rb = g.head_dim * elt;
  a.idx = idx;
  a.n_kept = n_kept;
  a.k = reinterpret_cast<const char*>(k);
  a.v = reinterpret_cast<const char*>(v);
  a.k_out = reinterpret_cast<char*>(k_out);
  a.v_out = reinterpret_cast<char*>(v_out);
  a.offs = seq_offsets(g);
  a.head_stride_bytes = g.kv_head_stride * elt;
  a.n_kv_heads = g.n_kv_heads;
  a.n_select = n_select;
  a.n_tail = n_tail;
  a.n_out = n_select + n_tail;
  if (a.n_out == 0) return hipSuccess;
  switch (rb) {
    case 128: return launch_rb<128>(a, g, st);
    case 256: return launch_rb<256>(a, g, st);
    case 512: return launch_rb<512>(a, g, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace dge
