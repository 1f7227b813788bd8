// Retention rules R_E (Alg. 1 step B): SnapKV max-pool + per-head top-B, and
// StreamingLLM sinks; optionally fused with the compaction (Alg. 1 step C).
//
// Top-B is an exact radix select on the float32 bit patterns of the pooled scores:
// scores are non-negative, so their IEEE bits order exactly like the values as
// unsigned integers.  Radix passes find the B'-th largest key T and how many keys equal
// to T must be kept; an ordered stream compaction then writes the kept positions in
// ascending order.  Taking tied keys in index order gives the lower-position tie-break
// directly, and the output needs no sort.
//
// Two kernels: select_topb_seg_kernel, the path for up to 32768 candidates per
// sequence (keys in registers, up to three passes of 12-14/10/9-7 bits, one workgroup
// per (replica, KV head, sequence, layer)); and select_topb_kernel, the fallback beyond
// it (keys in a global workspace, four 8-bit passes, one workgroup per (KV head,
// sequence), ordered compaction by wavefront ballots and a scan per 1024-key tile).
#include <type_traits>
#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int kSelThreads = 1024;
constexpr int kSelWaves = kSelThreads / kWave;
constexpr int kMaxLayers = 64;   // layers per multi-layer launch

struct SelectArgs {
  const float* scores;
  uint32_t* keys;        // workspace [batch][H_kv][key_stride]
  int32_t* idx;          // [batch][H_kv][n_select]
  int32_t* n_kept;       // [batch]
  SeqOffsets offs;
  int64_t total_rows;
  int64_t key_stride;
  int n_kv_heads, batch, pool_half, n_tail, n_select;
  // fused compaction (k_out == nullptr: selection only)
  const char* k;
  const char* v;
  char* k_out;
  char* v_out;
  int64_t head_stride_bytes;
  int row_bytes, n_out, replicas, rows_per_rep;
  // Several layers of a layer-major cache in one launch (segment kernel only): layer l
  // reads score/K/V heads [l*H_kv, (l+1)*H_kv), selects lay_nsel[l] rows and writes its
  // idx block at lay_idx_off[l] (int32 elements), n_kept at l*batch and its compacted
  // rows at row lay_out_off[l] of k_out / v_out.  One layer: n_layers = 1, offsets 0.
  int n_layers;
  int32_t lay_nsel[kMaxLayers];
  int64_t lay_idx_off[kMaxLayers];
  int64_t lay_out_off[kMaxLayers];
};

constexpr int kPoolHalo = 8;   // register path handles pool kernels up to 2*8+1

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
    int tie_before = 0, kept_before = 0, tot_gt = 0, tot_tie = 0;
    for (int w = 0; w < kSelWaves; ++w) {
      const int cg = cnt_gt[par][w], ct = cnt_tie[par][w];
      // ties of wave w that are still within the quota
      const int room = need - (tie_base + tot_tie);
      const int kt = room <= 0 ? 0 : (ct < room ? ct : room);
      if (w < wv) { tie_before += ct; kept_before += cg + kt; }
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

// Fast path for C <= THREADS * KPT.  Thread t owns the KPT consecutive candidates
// [t*KPT, (t+1)*KPT): their pooled keys stay in registers through the radix passes, and
// one workgroup-wide exclusive scan of (greater, tied) counts gives every thread the
// output position of its first kept candidate, so kept indices come out ascending
// without a sort.
//
// With `a.k_out` set, the workgroup also performs the compaction of its slice of
// output rows (replica `rep` of `a.replicas` per head): every replica repeats the
// selection (cheap, from L2) and copies rows [rep*rows_per_rep, (rep+1)*rows_per_rep)
// of [kept rows || tail || zero rows], so the row copies of one head spread over
// several compute units.

// Staging layout of the generic pool radius (up to kPoolHalo): candidate j at
// stage_pos(j + kPoolHalo), one pad word every 16 so that consecutive segments of the
// threads fall in different banks.
__host__ __device__ constexpr int stage_pos(int j) { return j + (j >> 4); }

// Staging layout of pool radius 2 and 3 (pool kernels 5 and 7): thread t's KPT
// candidates fill slot t+1 of kSlot words; slot 0 and slot THREADS+1 provide the zero
// halo of the first and the last thread.  A slot is a whole number of 16-byte units and
// that number is odd, so the 16-byte reads of eight consecutive lanes hit distinct banks.
template <int KPT>
struct PoolSlots {
  static constexpr int kSlot = ((KPT + 4) / 4) % 2 == 1 ? KPT + 4 : KPT + 8;
};

constexpr int kLdsBytesMax = 160 * 1024;
constexpr int kSegStaticLds = 512;   // scan and digit slots

// Dynamic LDS of one segment-kernel instance: the staging buffer and the three radix
// histograms (first digit: 12 bits, 16 bins per binade, up to 4096 candidates; 14 bits,
// 64 bins per binade, beyond, so that scores clustered in a few binades do not pile
// their atomics onto a few LDS addresses; then 10 bits and the rest).  The histograms
// sit beside the staging buffer when both fit, so they are cleared before the first
// barrier; otherwise they reuse the staging buffer once the pooled keys are in registers.
template <int THREADS, int KPT, int PH>
struct SegLds {
  static constexpr int kBits0 = THREADS * KPT > 4096 ? 14 : 12;
  static constexpr int kBits1 = 10;
  static constexpr int kBits2 = 31 - kBits0 - kBits1;
  static constexpr int kHistWords = (1 << kBits0) + (1 << kBits1) + (1 << kBits2);
  static constexpr int kStageWords = PH > 0 ? (THREADS + 2) * PoolSlots<KPT>::kSlot
                                            : stage_pos(THREADS * KPT + 2 * kPoolHalo) + 1;
  static constexpr bool kApart =
      (size_t)4 * ((kStageWords + 3) / 4 * 4 + kHistWords) + kSegStaticLds <= kLdsBytesMax;
  static constexpr int kHistOff = kApart ? (kStageWords + 3) / 4 * 4 : 0;
  static constexpr size_t kBytes =
      (size_t)4 * (kApart ? kHistOff + kHistWords
                          : (kStageWords > kHistWords ? kStageWords : kHistWords));
};

// Inclusive scan over the 64 lanes of a wavefront under an associative operation with
// identity `id`: DPP row shifts by 1, 2, 4 and 8 within each row of 16 lanes, then the
// row broadcasts of lane 15 (into rows 1 and 3) and lane 31 (into rows 2 and 3).  Lanes
// without a source combine with the identity (the `old` operand).
template <class Op>
__device__ __forceinline__ uint32_t wave_incl_scan(uint32_t v, uint32_t id, Op op) {
  const int o = (int)id;
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(o, (int)v, 0x111, 0xf, 0xf, false));  // row_shr:1
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(o, (int)v, 0x112, 0xf, 0xf, false));  // row_shr:2
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(o, (int)v, 0x114, 0xf, 0xf, false));  // row_shr:4
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(o, (int)v, 0x118, 0xf, 0xf, false));  // row_shr:8
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(o, (int)v, 0x142, 0xa, 0xf, false));  // row_bcast:15
  v = op(v, (uint32_t)__builtin_amdgcn_update_dpp(o, (int)v, 0x143, 0xc, 0xf, false));  // row_bcast:31
  return v;
}
struct OpAdd { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a + b; } };
struct OpMin { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a < b ? a : b; } };
struct OpMax { __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a > b ? a : b; } };

// Workgroup-wide exclusive prefix sum of one int per thread (one barrier).  Counts here
// stay below 2^16 per half, so two counters can share one packed word.
template <int THREADS>
__device__ __forceinline__ uint32_t block_excl_scan(uint32_t x, uint32_t* sh) {
  constexpr int WAVES = THREADS / kWave;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const uint32_t inc = wave_incl_scan(x, 0u, OpAdd());
  if (lane == 63) sh[wv] = inc;
  __syncthreads();
  uint32_t before = 0;
#pragma unroll
  for (int w = 0; w < WAVES; ++w)
    if (w < wv) before += sh[w];
  return before + inc - x;
}

// block_excl_scan of x that also reduces lo (minimum) and hi (maximum) over the
// workgroup in the same barrier; sh holds 3 * WAVES words.
template <int THREADS>
__device__ __forceinline__ uint32_t block_excl_scan_minmax(uint32_t x, uint32_t& lo, uint32_t& hi,
                                                           uint32_t* sh) {
  constexpr int WAVES = THREADS / kWave;
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  const uint32_t inc = wave_incl_scan(x, 0u, OpAdd());
  const uint32_t wlo = wave_incl_scan(lo, 0xffffffffu, OpMin());
  const uint32_t whi = wave_incl_scan(hi, 0u, OpMax());
  if (lane == 63) {
    sh[wv] = inc;
    sh[WAVES + wv] = wlo;
    sh[2 * WAVES + wv] = whi;
  }
  __syncthreads();
  uint32_t before = 0;
  lo = 0xffffffffu;
  hi = 0u;
#pragma unroll
  for (int w = 0; w < WAVES; ++w) {
    if (w < wv) before += sh[w];
    lo = min(lo, sh[WAVES + w]);
    hi = max(hi, sh[2 * WAVES + w]);
  }
  return before + inc - x;
}

// Find the digit d of a histogram of NB bins at which the count from the top first
// reaches `remaining`: above(d) < remaining <= above(d) + hist[d], above(d) = sum of the
// bins above d.  Thread t holds bin group (THREADS-1-t) in registers (16-byte LDS reads
// when the group spans 4 or more bins), so an ordinary prefix sum over the threads
// counts the keys above each group.  Writes {d, above(d), hist[d]} to out[0..2]; ends
// with a barrier, so every thread can read them.
template <int THREADS, int NB>
__device__ __forceinline__ void radix_find_digit(const uint32_t* hist, int remaining,
                                                uint32_t* scan_sh, int* out) {
  constexpr int PER = NB >= THREADS ? NB / THREADS : 1;
  const int grp = THREADS - 1 - (int)threadIdx.x;
  const int b0 = grp * PER;
  uint32_t c[PER];
  if constexpr (PER % 4 == 0) {
#pragma unroll
    for (int i = 0; i < PER; i += 4) {
      const uint4 v = *reinterpret_cast<const uint4*>(hist + b0 + i);
      c[i] = v.x; c[i + 1] = v.y; c[i + 2] = v.z; c[i + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int i = 0; i < PER; ++i) c[i] = b0 < NB ? hist[b0 + i] : 0u;
  }
  uint32_t cnt = 0;
#pragma unroll
  for (int i = 0; i < PER; ++i) cnt += c[i];
  uint32_t above = block_excl_scan<THREADS>(cnt, scan_sh);
  if (cnt > 0) {
#pragma unroll
    for (int i = PER - 1; i >= 0; --i) {
      if (above < (uint32_t)remaining && above + c[i] >= (uint32_t)remaining) {
        out[0] = b0 + i;
        out[1] = (int)above;
        out[2] = (int)c[i];
      }
      above += c[i];
    }
  }
  __syncthreads();
}

// One radix pass over the BITS-bit digit at SHIFT of the keys that match `prefix` under
// `mask`: histogram (LDS atomics into a cleared histogram), then the digit holding the
// remaining-th largest key.  Returns true when that digit's bin holds exactly the keys
// still to take: every key of the bin is kept, and the lower bits need no more passes.
template <int THREADS, int KPT, int BITS, int SHIFT>
__device__ __forceinline__ bool radix_pass(const uint32_t (&key)[KPT], int base, int C,
                                           uint32_t* hist, uint32_t* scan_sh, int* dig,
                                           uint32_t& prefix, uint32_t& mask, int& remaining) {
  constexpr int NB = 1 << BITS;
#pragma unroll
  for (int i = 0; i < KPT; ++i) {
    const bool in = base + i < C && (key[i] & mask) == prefix;
    if (in) atomicAdd(&hist[(key[i] >> SHIFT) & (uint32_t)(NB - 1)], 1u);
  }
  __syncthreads();
  radix_find_digit<THREADS, NB>(hist, remaining, scan_sh, dig);
  remaining -= dig[1];
  prefix |= (uint32_t)dig[0] << SHIFT;
  mask |= (uint32_t)(NB - 1) << SHIFT;
  return dig[2] == remaining;
}

template <int THREADS>
__device__ __forceinline__ void clear_words(uint32_t* p, int n) {
  for (int i = 4 * (int)threadIdx.x; i < n; i += 4 * THREADS)
    *reinterpret_cast<uint4*>(p + i) = make_uint4(0, 0, 0, 0);
}

// PH: max-pool radius fixed at compile time (2 or 3: kernels 5 and 7), or 0 for any
// radius up to kPoolHalo read from the arguments.
template <int THREADS, int KPT, int PH>
__global__ __launch_bounds__(THREADS) void select_topb_seg_kernel(SelectArgs a) {
  using Lds = SegLds<THREADS, KPT, PH>;
  constexpr int WAVES = THREADS / kWave;
  static_assert(KPT <= 32, "a thread keeps at most 32 pooled keys in registers");
  extern __shared__ __attribute__((aligned(16))) float stage[];
  const int per_layer = a.replicas * a.n_kv_heads * a.batch;
  const int units = per_layer * a.n_layers;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int layer = unit / per_layer, lu = unit - layer * per_layer;
  const int rep = lu % a.replicas, h = (lu / a.replicas) % a.n_kv_heads,
            b = lu / (a.replicas * a.n_kv_heads);
  const int hh = layer * a.n_kv_heads + h;   // head of the layer-major scores, K and V
  const int n_select = a.lay_nsel[layer];
  const int n_out = n_select + a.n_tail;
  const int tid = threadIdx.x;
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int C = N - a.n_tail;
  const int nsel = max(0, min(n_select, C));
  const bool writer = rep == 0;
  int32_t* out = a.idx + a.lay_idx_off[layer] + ((int64_t)b * a.n_kv_heads + h) * n_select;
  if (writer && h == 0 && tid == 0) a.n_kept[layer * a.batch + b] = nsel;
  if (writer)
    for (int r = nsel + tid; r < n_select; r += THREADS) out[r] = -1;
  uint32_t* const hist0 = reinterpret_cast<uint32_t*>(stage) + Lds::kHistOff;
  uint32_t* const hist1 = hist0 + (1 << Lds::kBits0);
  uint32_t* const hist2 = hist1 + (1 << Lds::kBits1);
  // the kept candidates in output order, written over the staging buffer (and the
  // histograms on top of it) once those are dead; nsel <= C <= THREADS * KPT words
  int32_t* const sel = reinterpret_cast<int32_t*>(stage);
  __shared__ uint32_t scan_sh[3 * WAVES];
  __shared__ int sh_digit[3][4];
  const int r0 = rep * a.rows_per_rep;
  const int r1 = min(n_out, r0 + a.rows_per_rep);
  const bool keep_all = nsel == C;

  if (keep_all) {
    // every candidate is kept, in order
    if (writer)
      for (int r = tid; r < C; r += THREADS) out[r] = r;
  } else if (nsel > 0) {
    const float* src = a.scores + (int64_t)hh * a.total_rows + s0;
    const int base = tid * KPT;
    if constexpr (Lds::kApart) clear_words<THREADS>(hist0, Lds::kHistWords);
    uint32_t key[KPT];
    bool staged = true;   // a barrier has followed the histogram clearing
    if constexpr (PH > 0) {
      // all of this thread's staging loads in flight at once, then the LDS stores into
      // the slot layout (candidates past C are zeros: scores are non-negative, so a zero
      // inside a window never changes its maximum)
      constexpr int S = PoolSlots<KPT>::kSlot;
      float sv[KPT];
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        const int j = tid + THREADS * i;
        sv[i] = j < C ? src[j] : 0.0f;
      }
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        const int j = tid + THREADS * i;
        stage[(j / KPT + 1) * S + j % KPT] = sv[i];
      }
      if (tid < 8) stage[tid < 4 ? KPT - 4 + tid : (THREADS + 1) * S + tid - 4] = 0.0f;
      __syncthreads();
      // the segment and four values of halo on each side, in 16-byte reads
      float w[KPT + 8];
      const float4 lh = *reinterpret_cast<const float4*>(stage + tid * S + KPT - 4);
      w[0] = lh.x; w[1] = lh.y; w[2] = lh.z; w[3] = lh.w;
#pragma unroll
      for (int k = 0; k < KPT / 4; ++k) {
        const float4 o = *reinterpret_cast<const float4*>(stage + (tid + 1) * S + 4 * k);
        w[4 + 4 * k] = o.x; w[5 + 4 * k] = o.y; w[6 + 4 * k] = o.z; w[7 + 4 * k] = o.w;
      }
      const float4 rh = *reinterpret_cast<const float4*>(stage + (tid + 2) * S);
      w[KPT + 4] = rh.x; w[KPT + 5] = rh.y; w[KPT + 6] = rh.z; w[KPT + 7] = rh.w;
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        float m = w[i + 4];
#pragma unroll
        for (int q = 1; q <= PH; ++q) m = fmaxf(m, fmaxf(w[i + 4 - q], w[i + 4 + q]));
        key[i] = __float_as_uint(m) & 0x7fffffffu;
      }
    } else if (a.pool_half > 0) {
      // generic radius: candidate j at stage_pos(j + kPoolHalo), kPoolHalo zeros on each side
      float sv[KPT];
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        const int j = tid + THREADS * i;
        sv[i] = j < C ? src[j] : 0.0f;
      }
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        const int j = tid + THREADS * i;
        if (j < C) stage[stage_pos(j + kPoolHalo)] = sv[i];
      }
      if (tid < 2 * kPoolHalo)
        stage[stage_pos(tid < kPoolHalo ? tid : C + tid)] = 0.0f;
      __syncthreads();
      // the segment and a halo of kPoolHalo on each side; reads past the zero padding
      // are clamped into it
      const int last = C + 2 * kPoolHalo - 1;
      float w[KPT + 2 * kPoolHalo];
#pragma unroll
      for (int i = 0; i < KPT + 2 * kPoolHalo; ++i)
        w[i] = stage[stage_pos(min(base + i, last))];
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        float m = w[i + kPoolHalo];
#pragma unroll
        for (int q = 1; q <= kPoolHalo; ++q)
          if (q <= a.pool_half) m = fmaxf(m, fmaxf(w[i + kPoolHalo - q], w[i + kPoolHalo + q]));
        key[i] = __float_as_uint(m) & 0x7fffffffu;
      }
    } else {
#pragma unroll
      for (int i = 0; i < KPT; ++i)
        key[i] = base + i < C ? (__float_as_uint(src[base + i]) & 0x7fffffffu) : 0u;
      staged = false;
    }
    if constexpr (!Lds::kApart) {
      __syncthreads();                     // staging reads done: the buffer becomes hist
      clear_words<THREADS>(hist0, Lds::kHistWords);
      __syncthreads();
    } else {
      if (!staged) __syncthreads();
    }

    // radix passes over bits 30..0 (bit 31 is zero for non-negative scores), most
    // significant digit first, until the digit's bin holds exactly the keys still to take
    uint32_t prefix = 0, mask = 0x80000000u;
    int remaining = nsel;
    bool exact = radix_pass<THREADS, KPT, Lds::kBits0, 31 - Lds::kBits0>(
        key, base, C, hist0, scan_sh, sh_digit[0], prefix, mask, remaining);
    if (!exact)
      exact = radix_pass<THREADS, KPT, Lds::kBits1, Lds::kBits2>(
          key, base, C, hist1, scan_sh, sh_digit[1], prefix, mask, remaining);

    // (greater, tied) counts of this thread's segment under the current prefix, packed
    // into one scanned word (C <= 32768, so neither half overflows 16 bits)
    auto count_scan = [&](uint32_t& lo, uint32_t& hi, auto with_minmax) {
      uint32_t packed = 0;
      lo = 0xffffffffu;
      hi = 0u;
#pragma unroll
      for (int i = 0; i < KPT; ++i) {
        const bool valid = base + i < C;
        const uint32_t km = key[i] & mask;
        const bool eq = valid && km == prefix;
        packed += (valid && km > prefix) ? 1u : 0u;
        packed += eq ? (1u << 16) : 0u;
        if constexpr (decltype(with_minmax)::value) {
          lo = eq ? min(lo, key[i]) : lo;
          hi = eq ? max(hi, key[i]) : hi;
        }
      }
      if constexpr (decltype(with_minmax)::value)
        return block_excl_scan_minmax<THREADS>(packed, lo, hi, scan_sh);
      else
        return block_excl_scan<THREADS>(packed, scan_sh);
    };
    uint32_t lo = 0, hi = 1, before;
    if constexpr (THREADS * KPT <= 4096) {
      // small candidate sets: the count scan also finds the smallest and largest key of
      // the threshold's bin; equal keys (max-pool plateaus) are all the threshold and
      // need no third pass (measured faster only at these sizes)
      before = count_scan(lo, hi, std::true_type{});
      if (!exact && lo != hi) {
        radix_pass<THREADS, KPT, Lds::kBits2, 0>(key, base, C, hist2, scan_sh, sh_digit[2],
                                                 prefix, mask, remaining);
        before = count_scan(lo, hi, std::false_type{});
      }
    } else {
      if (!exact)
        radix_pass<THREADS, KPT, Lds::kBits2, 0>(key, base, C, hist2, scan_sh, sh_digit[2],
                                                 prefix, mask, remaining);
      before = count_scan(lo, hi, std::false_type{});
    }
    // kept: keys above the threshold prefix, and `need` of the keys on it (index order)
    const uint32_t thr = prefix;
    const int need = remaining;
    const int gt_before = (int)(before & 0xffffu), tie_before = (int)(before >> 16);
    // the kept candidates of the segment take consecutive output positions; ties are
    // kept in index order up to the quota.  The scan's barrier has retired every read of
    // the staging buffer and the histograms, so sel[] may overwrite them.
    int q = gt_before + min(tie_before, need);
    int trank = tie_before;
#pragma unroll
    for (int i = 0; i < KPT; ++i) {
      const bool valid = base + i < C;
      const uint32_t km = key[i] & mask;
      const bool gt = valid && km > thr;
      const bool eq = valid && km == thr;
      const bool keep = gt || (eq && trank < need);
      trank += eq ? 1 : 0;
      if (keep && q < nsel) sel[q] = base + i;
      q += keep ? 1 : 0;
    }
  }
  lds_barrier();                           // sel[] complete
  if (writer && !keep_all)
    for (int r = tid; r < nsel; r += THREADS) out[r] = sel[r];
  if (a.k_out == nullptr) return;

  // compaction of output rows [r0, r1): kept rows, then the tail, then zero rows; the
  // loads of kCopyBatch rows per thread are issued before their stores, so a thread
  // waits for one round trip per batch rather than per row
  constexpr int kCopyBatch = 4;
  const int tpr = a.row_bytes / 16;
  const int rpp = THREADS / tpr;
  const int part = tid % tpr;
  const int64_t obase = a.lay_out_off[layer] + ((int64_t)b * a.n_kv_heads + h) * n_out;
  for (int rb = r0 + tid / tpr; rb < r1; rb += kCopyBatch * rpp) {
    uint4 kv[kCopyBatch], vv[kCopyBatch];
#pragma unroll
    for (int u = 0; u < kCopyBatch; ++u) {
      const int r = rb + u * rpp;
      int srow = -1;
      if (r < r1) {
        if (r < nsel) srow = keep_all ? r : sel[r];
        else if (r < nsel + a.n_tail) srow = C + (r - nsel);
      }
      kv[u] = make_uint4(0, 0, 0, 0);
      vv[u] = make_uint4(0, 0, 0, 0);
      if (srow >= 0) {
        const int64_t in = hh * a.head_stride_bytes + (s0 + srow) * a.row_bytes + part * 16;
        kv[u] = load16(a.k + in);
        vv[u] = load16(a.v + in);
      }
    }
#pragma unroll
    for (int u = 0; u < kCopyBatch; ++u) {
      const int r = rb + u * rpp;
      if (r < r1) {
        const int64_t o = (obase + r) * a.row_bytes + part * 16;
        *reinterpret_cast<uint4*>(a.k_out + o) = kv[u];
        *reinterpret_cast<uint4*>(a.v_out + o) = vv[u];
      }
    }
  }
}

__global__ __launch_bounds__(256) void select_streaming_kernel(int32_t* idx, int32_t* n_kept,
                                                                SeqOffsets offs, int n_kv_heads,
                                                                int n_sink, int n_recent) {
  const int h = blockIdx.x, b = blockIdx.y;
  const int N = (int)(offs[b + 1] - offs[b]);
  const int C = N - n_recent;
  const int nk = min(n_sink, C > 0 ? C : 0);
  int32_t* out = idx + ((int64_t)b * n_kv_heads + h) * n_sink;
  for (int r = threadIdx.x; r < n_sink; r += blockDim.x) out[r] = r < nk ? r : -1;
  if (h == 0 && threadIdx.x == 0) n_kept[b] = nk;
}

template <int THREADS, int KPT, int PH>
hipError_t launch_seg_ph(const SelectArgs& a, dim3 grid, hipStream_t st) {
  constexpr size_t lds = SegLds<THREADS, KPT, PH>::kBytes;
  static_assert(lds + kSegStaticLds <= kLdsBytesMax, "segment kernel LDS");
  if (lds > 64 * 1024) {
    const hipError_t e = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&select_topb_seg_kernel<THREADS, KPT, PH>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e != hipSuccess) return e;
  }
  hipLaunchKernelGGL((select_topb_seg_kernel<THREADS, KPT, PH>), grid, dim3(THREADS), lds, st, a);
  return hipGetLastError();
}

template <int THREADS, int KPT>
hipError_t launch_seg(const SelectArgs& a, dim3 grid, hipStream_t st) {
  if (a.pool_half == 2) return launch_seg_ph<THREADS, KPT, 2>(a, grid, st);
  if (a.pool_half == 3) return launch_seg_ph<THREADS, KPT, 3>(a, grid, st);
  return launch_seg_ph<THREADS, KPT, 0>(a, grid, st);
}

SelectArgs make_args(const dge_geom_t& g, const float* scores, int pool_kernel, int n_tail,
                     int n_select, int32_t* idx, int32_t* n_kept, void* ws) {
  SelectArgs a{};
  a.scores = scores;
  a.keys = reinterpret_cast<uint32_t*>(ws);
  a.idx = idx;
  a.n_kept = n_kept;
  a.offs = seq_offsets(g);
  a.total_rows = total_rows(g);
  a.key_stride = (max_seq_rows(g) + 63) / 64 * 64;
  a.n_kv_heads = g.n_kv_heads;
  a.batch = g.batch;
  a.pool_half = pool_kernel / 2;
  a.n_tail = n_tail;
  a.n_select = n_select;
  a.n_out = n_select + n_tail;
  a.replicas = 1;
  a.rows_per_rep = n_select + n_tail > 0 ? n_select + n_tail : 1;
  a.n_layers = 1;
  a.lay_nsel[0] = n_select;
  a.lay_idx_off[0] = 0;
  a.lay_out_off[0] = 0;
  return a;
}

// Spread each head's row copies over enough replicas to occupy the chip while keeping
// the repeated selection bounded: at most 32 replicas of at least 32 rows each (at 8
// heads of 514 output rows, 17 replicas run 0.25 us faster than 9 of 64 rows).
void set_replicas(SelectArgs& a, int units, int n_out) {
  int reps = 256 / (units > 0 ? units : 1);
  const int by_rows = (n_out + 31) / 32;
  reps = reps > by_rows ? by_rows : reps;
  reps = reps > 32 ? 32 : reps;
  reps = reps < 1 ? 1 : reps;
  const int rpr = (n_out + reps - 1) / reps;
  a.replicas = reps;
  a.rows_per_rep = rpr > 0 ? rpr : 1;
}

// Launch the segment kernel when the largest candidate set fits; returns false when
// the global-memory fallback must be used.
bool launch_fast(const SelectArgs& a, const dge_geom_t& g, int64_t cmax, hipStream_t st,
                 hipError_t* err) {
  if (a.pool_half > kPoolHalo) return false;
  const dim3 grid(xcd_grid(a.replicas * g.n_kv_heads * g.batch * a.n_layers));
  // (threads, candidates per thread): more threads per workgroup shorten the serial
  // per-thread loops of every radix pass (measured best at each size on MI355X)
  if (cmax <= 1024) *err = launch_seg<256, 4>(a, grid, st);
  else if (cmax <= 2048) *err = launch_seg<256, 8>(a, grid, st);
  else if (cmax <= 4096) *err = launch_seg<512, 8>(a, grid, st);
  else if (cmax <= 8192) *err = launch_seg<1024, 8>(a, grid, st);
  else if (cmax <= 16384) *err = launch_seg<1024, 16>(a, grid, st);
  else if (cmax <= 32768) *err = launch_seg<1024, 32>(a, grid, st);
  else return false;
  return true;
}

}  // namespace

size_t select_workspace_bytes(const dge_geom_t& g) {
  return (size_t)g.batch * g.n_kv_heads * (size_t)((max_seq_rows(g) + 63) / 64 * 64) * 4 + 256;
}

hipError_t launch_select_topb(const dge_geom_t& g, const float* scores, int pool_kernel,
                              int n_tail, int n_select, int32_t* idx, int32_t* n_kept, void* ws,
                              hipStream_t st) {
  SelectArgs a = make_args(g, scores, pool_kernel, n_tail, n_select, idx, n_kept, ws);
  hipError_t err = hipSuccess;
  if (launch_fast(a, g, max_seq_rows(g) - n_tail, st, &err)) return err;
  hipLaunchKernelGGL(select_topb_kernel, dim3(g.n_kv_heads, g.batch), dim3(kSelThreads), 0, st, a);
  return hipGetLastError();
}

hipError_t launch_select_compact(const dge_geom_t& g, const float* scores, int pool_kernel,
                                 int n_tail, int n_select, int32_t* idx, int32_t* n_kept,
                                 const void* k, const void* v, void* k_out, void* v_out, void* ws,
                                 hipStream_t st) {
  SelectArgs a = make_args(g, scores, pool_kernel, n_tail, n_select, idx, n_kept, ws);
  const int elt = g.dtype == DGE_BF16 ? 2 : 4;
  a.k = reinterpret_cast<const char*>(k);
  a.v = reinterpret_cast<const char*>(v);
  a.k_out = reinterpret_cast<char*>(k_out);
  a.v_out = reinterpret_cast<char*>(v_out);
  a.head_stride_bytes = g.kv_head_stride * elt;
  a.row_bytes = g.head_dim * elt;
  set_replicas(a, g.batch * g.n_kv_heads, a.n_out);
  hipError_t err = hipSuccess;
  if (launch_fast(a, g, max_seq_rows(g) - n_tail, st, &err)) return err;
  // candidate sets beyond the register path: select, then the separate row gather
  a.k_out = nullptr;
  a.replicas = 1;
  hipLaunchKernelGGL(select_topb_kernel, dim3(g.n_kv_heads, g.batch), dim3(kSelThreads), 0, st, a);
  err = hipGetLastError();
  if (err != hipSuccess) return err;
  return launch_compact(g, idx, n_kept, n_select, n_tail, k, v, k_out, v_out, st);
}

hipError_t launch_select_compact_layers(const dge_geom_t& g, int n_layers, const float* scores,
                                        int pool_kernel, int n_tail, const int32_t* n_select_host,
                                        int32_t* idx, int32_t* n_kept, const void* k, const void* v,
                                        void* k_out, void* v_out, void* ws, hipStream_t st) {
  const int elt = g.dtype == DGE_BF16 ? 2 : 4;
  const int64_t heads = (int64_t)g.batch * g.n_kv_heads;
  const int64_t cmax = max_seq_rows(g) - n_tail;
  const int64_t hsz = (int64_t)g.n_kv_heads * g.kv_head_stride * elt;   // bytes per layer
  const int64_t ssz = (int64_t)g.n_kv_heads * total_rows(g);             // scores per layer
  const char* kc = static_cast<const char*>(k);
  const char* vc = static_cast<const char*>(v);
  char* koc = static_cast<char*>(k_out);
  char* voc = static_cast<char*>(v_out);
  const int row_bytes = g.head_dim * elt;
  int64_t io = 0, oo = 0;   // packed idx elements and output rows of the layers before
  if (pool_kernel / 2 <= kPoolHalo && cmax <= 32768) {
    // groups of up to kMaxLayers layers, one launch each
    for (int l0 = 0; l0 < n_layers; l0 += kMaxLayers) {
      const int nl = n_layers - l0 < kMaxLayers ? n_layers - l0 : kMaxLayers;
      int max_sel = 0;
      for (int l = 0; l < nl; ++l)
        max_sel = max_sel > n_select_host[l0 + l] ? max_sel : n_select_host[l0 + l];
      SelectArgs a = make_args(g, scores + l0 * ssz, pool_kernel, n_tail, max_sel, idx + io,
                               n_kept + (int64_t)l0 * g.batch, ws);
      a.k = kc + l0 * hsz;
      a.v = vc + l0 * hsz;
      a.k_out = koc + oo * row_bytes;
      a.v_out = voc + oo * row_bytes;
      a.head_stride_bytes = g.kv_head_stride * elt;
      a.row_bytes = row_bytes;
      a.n_layers = nl;
      int64_t gio = 0, goo = 0;
      for (int l = 0; l < nl; ++l) {
        a.lay_nsel[l] = n_select_host[l0 + l];
        a.lay_idx_off[l] = gio;
        a.lay_out_off[l] = goo;
        gio += heads * n_select_host[l0 + l];
        goo += heads * (n_select_host[l0 + l] + n_tail);
      }
      set_replicas(a, (int)(heads * nl), max_sel + n_tail);
      hipError_t err = hipSuccess;
      if (!launch_fast(a, g, cmax, st, &err)) return hipErrorInvalidValue;   // excluded above
      if (err != hipSuccess) return err;
      io += gio;
      oo += goo;
    }
    return hipSuccess;
  }
  // pool radius beyond the register halo or candidate sets beyond the register path:
  // one launch per layer on that layer's slices
  for (int l = 0; l < n_layers; ++l) {
    const int ns = n_select_host[l];
    const hipError_t err = launch_select_compact(
        g, scores + l * ssz, pool_kernel, n_tail, ns, idx + io, n_kept + (int64_t)l * g.batch,
        kc + l * hsz, vc + l * hsz, koc + oo * row_bytes, voc + oo * row_bytes, ws, st);
    if (err != hipSuccess) return err;
    io += heads * ns;
    oo += heads * (ns + n_tail);
  }
  return hipSuccess;
}

hipError_t launch_select_streaming(const dge_geom_t& g, int n_sink, int n_recent, int32_t* idx,
                                   int32_t* n_kept, hipStream_t st) {
  hipLaunchKernelGGL(select_streaming_kernel, dim3(g.n_kv_heads, g.batch), dim3(256), 0, st, idx,
                     n_kept, seq_offsets(g), g.n_kv_heads, n_sink, n_recent);
  return hipGetLastError();
}

}  // namespace dge
