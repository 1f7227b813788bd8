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

// In-place compaction: the compacted rows of (b, h) overwrite the first n_out = n_kept +
// n_tail rows of that head's own segment of the cache.  Output row r takes source row
// src(r) = idx[r] (r < n_kept) or C + (r - n_kept) (the tail); sources ascend with r and
// src(r) >= r, so rows only move down.  Only rows [0, n_out) are written, so a source at or
// above n_out is never overwritten: the rows whose source lies there ("far" rows) can be
// copied in any order by any number of workgroups.  The others ("near" rows, src(r) <
// n_out) form a prefix of the output rows, and their sources may be the destinations of
// other rows.  Two launches:
//   1. near rows, one workgroup per (KV head, sequence), in order: it reads every source
//      of a chunk of rows, meets a barrier, then writes the chunk (a chunk's rows lie below
//      every source of the later chunks, and the sources of this and the earlier chunks
//      were read before the barrier); it stops after the chunk whose successor starts with
//      a far row.
//      Typically the near prefix is short (the kept keys that already sit below n_out).
//   2. far rows, many workgroups per head, each thread loading the 16-byte pieces of
//      several rows before storing them.  Their sources (>= n_out) are never written,
//      their destinations [r*, n_out) are not read by this launch, and launch 1 read the
//      near rows' sources before any of them is overwritten.
constexpr int kInplaceThreads = 1024;
constexpr int kInplaceUnroll = 8;

// (launch 2) source of output row r, -1 past the compacted rows
__device__ __forceinline__ int inplace_src(const int32_t* ix, int r, int nk, int C, int n_out) {
  if (r < nk) return max(r, min(ix[r], C - 1));   // a malformed index never moves a row up
  if (r < n_out) return C + (r - nk);
  return -1;
}

template <int RB>
__global__ __launch_bounds__(kInplaceThreads) void compact_inplace_near_kernel(CompactArgs a,
                                                                              char* k, char* v) {
  constexpr int TPR = RB / 16;                    // threads per row
  constexpr int RPP = kInplaceThreads / TPR;      // rows per pass
  constexpr int CHUNK = RPP * kInplaceUnroll;     // rows read before each barrier
  const int h = blockIdx.x, b = blockIdx.y;
  const int sub = threadIdx.x / TPR, part = threadIdx.x % TPR;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int C = N - a.n_tail;
  const int32_t* ix = a.idx + ((int64_t)b * a.n_kv_heads + h) * a.n_select;
  const int64_t base = h * a.head_stride_bytes + s0 * RB + part * 16;
  // the indices are loaded for every r < n_select without waiting for n_kept (a chain
  // of dependent round trips is what this launch costs); n_kept then picks index or tail
  auto index_at = [&](int r) { return r < a.n_select ? ix[r] : 0; };
  const int nk_raw = a.n_kept[b];
  for (int c0 = 0;; c0 += CHUNK) {
    int iv[kInplaceUnroll];
#pragma unroll
    for (int u = 0; u < kInplaceUnroll; ++u) iv[u] = index_at(c0 + u * RPP + sub);
    const int iv_next = index_at(c0 + CHUNK);     // first row of the next chunk
    const int nk = max(0, min(nk_raw, min(a.n_select, C)));
    const int n_out = nk + a.n_tail;
    auto src_of = [&](int r, int i) {
      if (r < nk) return max(r, min(i, C - 1));   // a malformed index never moves a row up
      if (r < n_out) return C + (r - nk);
      return -1;
    };
    uint4 kv[kInplaceUnroll], vv[kInplaceUnroll];
    int src[kInplaceUnroll];
#pragma unroll
    for (int u = 0; u < kInplaceUnroll; ++u) {
      const int r = c0 + u * RPP + sub;
      const int sr = src_of(r, iv[u]);
      // far rows are left to launch 2, rows already in place are not copied
      src[u] = (sr >= 0 && sr < n_out && sr != r) ? sr : -1;
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
    // sources ascend, so once the next chunk's first row is not near, no later row is;
    // the decision is the same in every thread
    const int s_next = src_of(c0 + CHUNK, iv_next);
    if (c0 + CHUNK >= n_out || s_next < 0 || s_next >= n_out) break;
  }
}

constexpr int kFarRows = 4;     // rows per thread in launch 2

template <int RB>
__global__ __launch_bounds__(256) void compact_inplace_far_kernel(CompactArgs a, char* k, char* v) {
  constexpr int TPR = RB / 16;
  constexpr int RPB = 256 / TPR;                  // rows per pass of the workgroup
  const int h = blockIdx.y, b = blockIdx.z;
  const int sub = threadIdx.x / TPR, part = threadIdx.x % TPR;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int C = N - a.n_tail;
  const int nk = max(0, min(a.n_kept[b], min(a.n_select, C)));
  const int n_out = nk + a.n_tail;
  const int r0 = blockIdx.x * (RPB * kFarRows);
  if (r0 >= n_out) return;
  const int32_t* ix = a.idx + ((int64_t)b * a.n_kv_heads + h) * a.n_select;
  const int64_t base = h * a.head_stride_bytes + s0 * RB + part * 16;
  int src[kFarRows];
  uint4 kv[kFarRows], vv[kFarRows];
#pragma unroll
  for (int u = 0; u < kFarRows; ++u) {
    const int r = r0 + u * RPB + sub;
    const int s = inplace_src(ix, r, nk, C, n_out);
    src[u] = s >= n_out ? s : -1;                 // far rows only
  }
#pragma unroll
  for (int u = 0; u < kFarRows; ++u)
    if (src[u] >= 0) {
      kv[u] = load16(k + base + (int64_t)src[u] * RB);
      vv[u] = load16(v + base + (int64_t)src[u] * RB);
    }
#pragma unroll
  for (int u = 0; u < kFarRows; ++u)
    if (src[u] >= 0) {
      const int r = r0 + u * RPB + sub;
      *reinterpret_cast<uint4*>(k + base + (int64_t)r * RB) = kv[u];
      *reinterpret_cast<uint4*>(v + base + (int64_t)r * RB) = vv[u];
    }
}

template <int RB>
hipError_t launch_inplace_rb(const CompactArgs& a, const dge_geom_t& g, char* k, char* v,
                             hipStream_t st) {
  constexpr int RPB = 256 / (RB / 16);
  hipLaunchKernelGGL((compact_inplace_near_kernel<RB>), dim3(g.n_kv_heads, g.batch),
                     dim3(kInplaceThreads), 0, st, a, k, v);
  const dim3 grid((a.n_out + RPB * kFarRows - 1) / (RPB * kFarRows), g.n_kv_heads, g.batch);
  hipLaunchKernelGGL((compact_inplace_far_kernel<RB>), grid, dim3(256), 0, st, a, k, v);
  return hipGetLastError();
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
  if (a.n_out == 0) return hipSuccess;
  switch (rb) {
    case 128: return launch_inplace_rb<128>(a, g, kc, vc, st);
    case 256: return launch_inplace_rb<256>(a, g, kc, vc, st);
    case 512: return launch_inplace_rb<512>(a, g, kc, vc, st);
    default: return hipErrorInvalidValue;
  }
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
