// Retention rules R_E (Alg. 1 step B): SnapKV max-pool + per-head top-B, and
// StreamingLLM sinks.  One workgroup per (sequence, KV head).
//
// Top-B is an exact radix select on the float32 bit patterns of the pooled scores:
// scores are non-negative, so their IEEE bits order exactly like the values as
// unsigned integers.  Four 8-bit passes find the B'-th largest key T and how many
// keys equal to T must be kept; an ordered stream compaction (wavefront ballots +
// a workgroup scan per 1024-key tile) then writes the kept positions in ascending
// order.  Taking tied keys in index order gives the lower-position tie-break
// directly, and the output needs no sort.
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;

struct SelectArgs {
  const float* scores;
  uint32_t* keys;        // workspace [batch][H_kv][key_stride]
  int32_t* idx;          // [batch][H_kv][n_select]
  int32_t* n_kept;       // [batch]
  const int64_t* offs;
  int64_t total_rows;
  int64_t key_stride;
  int n_kv_heads, pool_half, n_tail, n_select;
};

__global__ __launch_bounds__(kSelThreads) void select_topb_kernel(SelectArgs a) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int C = N - a.n_tail;
  const int nsel = min(a.n_select, C);
  int32_t* out = a.idx + ((int64_t)b * a.n_kv_heads + h) * a.n_select;
  if (h == 0 && tid == 0) a.n_kept[b] = nsel;
  for (int r = nsel + tid; r < a.n_select; r += kSelThreads) out[r] = -1;
  if (nsel <= 0) return;
  if (nsel == C) {   // budget covers every candidate: keep all, in order
    for (int r = tid; r < C; r += kSelThreads) out[r] = r;
    return;
  }

  // 1-D max-pool over the candidates only, written as radix keys
  const float* src = a.scores + (int64_t)h * a.total_rows + s0;
  uint32_t* keys = a.keys + ((int64_t)b * a.n_kv_heads + h) * a.key_stride;
  for (int j = tid; j < C; j += kSelThreads) {
    const int lo = max(0, j - a.pool_half), hi = min(C - 1, j + a.pool_half);
    float v = src[lo];
    for (int i = lo + 1; i <= hi; ++i) v = fmaxf(v, src[i]);
    keys[j] = __float_as_uint(v);
  }
  __syncthreads();

  __shared__ uint32_t hist[256];
  __shared__ uint32_t sh_digit, sh_above;
  if (tid == 0) { sh_digit = 0; sh_above = 0; }
  uint32_t prefix = 0, mask = 0;
  int remaining = nsel;   // keys still to take at or below the current prefix
  for (int shift = 24; shift >= 0; shift -= 8) {
    if (tid < 256) hist[tid] = 0;
    __syncthreads();
    for (int j = tid; j < C; j += kSelThreads) {
      const uint32_t key = keys[j];
      if ((key & mask) == prefix) atomicAdd(&hist[(key >> shift) & 255u], 1u);
    }
    __syncthreads();
    if (wv == 0) {
      // lane l owns digits 4l..4l+3; find the digit where the count from the top
      // first reaches `remaining`
      uint32_t c[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) c[i] = hist[4 * lane + i];
      const uint32_t tot = c[0] + c[1] + c[2] + c[3];
      uint32_t suf = tot;   // inclusive suffix sum over lanes >= l
#pragma unroll
      for (int o = 1; o < 64; o <<= 1) {
        const uint32_t v = __shfl_down(suf, o, 64);
        if (lane + o < 64) suf += v;
      }
      uint32_t above = suf - tot;   // keys with a digit above this lane's four
#pragma unroll
      for (int i = 3; i >= 0; --i) {
        if (above < (uint32_t)remaining && above + c[i] >= (uint32_t)remaining) {
          sh_digit = 4 * lane + i;
          sh_above = above;
        }
        above += c[i];
      }
    }
    __syncthreads();
    remaining -= (int)sh_above;
    prefix |= sh_digit << shift;
    mask |= 255u << shift;
    __syncthreads();
  }
  const uint32_t thr = prefix;     // the nsel-th largest key
  const int need = remaining;      // keys equal to thr that are kept (>= 1)

  __shared__ int cnt_gt[2][kSelWaves], cnt_tie[2][kSelWaves];
  int kept_base = 0, tie_base = 0;
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));
  for (int t0 = 0, par = 0; t0 < C; t0 += kSelThreads, par ^= 1) {
    const int j = t0 + tid;
    const uint32_t key = j < C ? keys[j] : 0u;
    const bool gt = j < C && key > thr;
    const bool tie = j < C && key == thr;
    const uint64_t mg = __ballot(gt), mt = __ballot(tie);
    if (lane == 0) {
      cnt_gt[par][wv] = __popcll(mg);
      cnt_tie[par][wv] = __popcll(mt);
    }
    __syncthreads();
    int gt_before = 0, tie_before = 0, kept_before = 0, tot_gt = 0, tot_tie = 0;
    for (int w = 0; w < kSelWaves; ++w) {
      const int cg = cnt_gt[par][w], ct = cnt_tie[par][w];
      // ties of wave w that are still within the quota
      const int room = need - (tie_base + tot_tie);
      const int kt = room <= 0 ? 0 : (ct < room ? ct : room);
      if (w < wv) { gt_before += cg; tie_before += ct; kept_before += cg + kt; }
      tot_gt += cg;
      tot_tie += ct;
    }
    const int tie_rank = tie_base + tie_before + __popcll(mt & lt_mask);
    const bool keep = gt || (tie && tie_rank < need);
    const uint64_t mk = __ballot(keep);
    const int pos = kept_base + kept_before + __popcll(mk & lt_mask);
    if (keep && pos < nsel) out[pos] = j;
    const int tie_taken = min(tot_tie, max(0, need - tie_base));
    kept_base += tot_gt + tie_taken;
    tie_base += tot_tie;
  }
}

__global__ __launch_bounds__(256) void select_streaming_kernel(int32_t* idx, int32_t* n_kept,
                                                                const int64_t* offs, int n_kv_heads,
                                                                int n_sink, int n_recent) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int N = (int)(offs[b + 1] - offs[b]);
  const int C = N - n_recent;
  const int nk = min(n_sink, C > 0 ? C : 0);
  int32_t* out = idx + ((int64_t)b * n_kv_heads + h) * n_sink;
  for (int r = threadIdx.x; r < n_sink; r += blockDim.x) out[r] = r < nk ? r : -1;
  if (h == 0 && threadIdx.x == 0) n_kept[b] = nk;
}

}  // namespace

size_t select_workspace_bytes(const dge_geom_t& g) {
  return (size_t)g.batch * g.n_kv_heads * (size_t)((max_seq_rows(g) + 63) / 64 * 64) * 4 + 256;
}

hipError_t launch_select_topb(const dge_geom_t& g, const float* scores, int pool_kernel,
                              int n_tail, int n_select, int32_t* idx, int32_t* n_kept, void* ws,
                              hipStream_t st) {
  SelectArgs a{};
  a.scores = scores;
  a.keys = reinterpret_cast<uint32_t*>(ws);
  a.idx = idx;
  a.n_kept = n_kept;
  a.offs = g.kv_offsets;
  a.total_rows = total_rows(g);
  a.key_stride = (max_seq_rows(g) + 63) / 64 * 64;
  a.n_kv_heads = g.n_kv_heads;
  a.pool_half = pool_kernel / 2;
  a.n_tail = n_tail;
  a.n_select = n_select;
  hipLaunchKernelGGL(select_topb_kernel, dim3(g.n_kv_heads, g.batch), dim3(kSelThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_select_streaming(const dge_geom_t& g, int n_sink, int n_recent, int32_t* idx,
                                   int32_t* n_kept, hipStream_t st) {
  hipLaunchKernelGGL(select_streaming_kernel, dim3(g.n_kv_heads, g.batch), dim3(256), 0, st, idx,
                     n_kept, g.kv_offsets, g.n_kv_heads, n_sink, n_recent);
  return hipGetLastError();
}

}  // namespace dge
