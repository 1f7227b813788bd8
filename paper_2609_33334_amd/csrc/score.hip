// Window / draft scoring of every cached key (Alg. 1 step B; App. "Diagnostic details").
//
//   raw[h][j] = (1/G) sum_{g in group h} sum_r softmax_j(q_{g,r} . k_j / sqrt(d)),
//   softmax over keys j <= p_r (causal), fp32 after the bf16/fp32 product.
//
// A column sum needs every scoring row's global normaliser first, so one layer runs
// as three launches over the same split of the keys into chunks:
//   1. stats : each workgroup streams its chunk of K and keeps, per query row, the
//              running (max, sum of 2^(x - max)) of its logits (log2 domain), stored
//              as one log2-sum-exp per row and chunk;
//   2. reduce: the chunk partials of every (row, sequence, KV head) merge into
//              c_r = log2 Z_r (a lane per row when there are few chunks, else a
//              wavefront per row);
//   3. colsum: each workgroup streams its chunk again, P = 2^(x - c_r), sums over all
//              rows of the group and writes raw[] (the K slab of one layer, 8-34 MB at
//              Llama-3-8B geometry, is still in the 256 MB Infinity Cache).
// With caller-supplied row LSEs (dge_score_lse) only the colsum pass runs.
// (Measured slower on MI355X, and not used: a single launch that waits in-kernel for
// the other chunks of a head -- device-scope atomics and coherent loads cost
// microseconds each -- and merging the chunk partials inside every colsum workgroup,
// whose extra loads join the burst of query and K loads at kernel start.)
//
// Workgroups are laid out XCD-aware (see xcd_unit): the chunks of one KV head share an
// XCD, so its query block is fetched into one L2, and the colsum pass finds each chunk
// in the L2 that streamed it during the stats pass.
//
// Work split inside a workgroup (4 wavefronts, one KV head, one chunk of keys):
// - The G * n_rows query rows form T 16-row tiles.  Each wavefront owns T/4 of them
//   for every key and takes the T%4 leftover tiles only for its own 16-key subtile of
//   each K tile (see slot_tile), so the four wavefronts do equal work and none computes
//   a padding tile.  Query fragments stay in registers for the whole chunk (48 VGPRs at
//   Llama-3-8B geometry), so two stats workgroups (three colsum ones) fit on a compute
//   unit.
// - Each 64-key tile of K is copied from HBM straight into LDS (global_load_lds, 16
//   bytes per lane, a row per 16 lanes) with the 16-byte units of row r XOR-swizzled
//   by r, so the 16 lanes that read one fragment column hit 16 different bank groups.
//   Three tiles are always in flight (a 4-stage ring of 16 KB buffers; two with three
//   workgroups per compute unit; dummy copies past the end of a chunk keep every wait
//   count fixed) while one is on the matrix cores; the loop's barriers wait on LDS
//   traffic only, so the copies are never drained early.
// - Tile bodies are branch-free: all products of a tile (or of a group of subtiles)
//   are issued before their results are used, so the exp2 work overlaps the matrix
//   cores; a separate masked body runs only where a tile reaches past the first
//   scoring position.
// - stats uses the transposed product (A = keys, B = query rows): a lane then holds
//   4 keys of ONE row, so the per-row max/sum is in-lane (one running-max update per
//   group of subtiles) and needs cross-lane steps only at the end of the chunk.
// - colsum uses A = query rows, B = keys: a lane holds 4 rows of ONE key, the sum
//   over rows is in-lane, then across the 4 lane groups (permlane swaps) and the 4
//   wavefronts (LDS, double-buffered, flushed after the next tile's barrier).
// On long walks at Llama-3-8B geometry (bf16, d = 128, 8 or 9 row tiles) both passes
// instead give each wavefront every row tile and its own run of 16-key subtiles through
// a private ring, with no barrier in the loop (score_stats_wave_kernel,
// score_colsum_wave_kernel): under the passes' arithmetic on random operands the
// per-tile barrier of the shared ring slows the K stream.
#include <type_traits>

#include "dge_device.hpp"
#include "dge_internal.hpp"

namespace dge {
namespace {

constexpr int KT = 64;          // keys per workgroup iteration
constexpr int kThreads = 256;

struct ScoreArgs {
  const void* q;
  const void* k;
  float* raw;
  float* partial;    // [batch][H_kv][n_chunks][M_pad] log2-sum-exp of each row per chunk
  float* rowc;       // [batch][H_kv][M_pad]  log2 of each row's softmax normaliser
  const float* lse_in;      // optional [H_q][batch * n_rows] natural-log row LSE
  float* lse_out;           // optional output: the merged row LSE, natural log, same layout
  SeqOffsets offs;
  int64_t kv_head_stride;   // elements
  int64_t q_head_stride;    // elements between query heads = batch * n_rows * D
  int64_t total_rows;       // T
  int n_kv_heads, batch, G, n_rows, p0_from_end;
  int M, M_pad, n_tiles, groups, iters, chunk_keys, n_chunks;
  int c_iters, c_chunk_keys, c_n_chunks;   // the colsum pass's split of the keys
  float scale_log2;         // log2(e) / sqrt(d)
  float inv_G;
};

template <typename T, int D>
struct KTile {
  static constexpr int kRowBytes = D * Elem<T>::kBytes;
  static constexpr int kUnits = kRowBytes / 16;                // 16-byte units per row
  static constexpr int kInstr = KT * kUnits / kThreads;        // copy instructions per wave
  static constexpr int kBytes = KT * kRowBytes;
};

// Global->LDS copy of one 64-key tile, issued by all 4 wavefronts: wavefront w's
// instruction i fills bytes [(w*kInstr + i) KB, +1 KB) of the tile, lane l the 16 bytes
// at offset 16*l of that kilobyte.  Each lane fetches the global unit that belongs at
// its LDS position under the XOR swizzle (unit u of row r at position u ^ (r % kUnits)),
// so a fragment read later hits 16 different bank groups.  The lane's row and column
// within a tile (KCopy) are computed once; a copy is then a wave-uniform base plus a
// 32-bit lane offset whose row is clamped to the sequence's last row (their logits are
// masked).  A dummy copy (real == false) reads tile 0 of the sequence again: it keeps
// the number of copies in flight constant at the end of a chunk, so that every wait
// below has a fixed count, and hits the cache.  Nothing here branches, so every path
// through the kernel issues the same copies.
template <typename T, int D>
struct KCopy {
  using KTl = KTile<T, D>;
  uint32_t row[KTl::kInstr];     // row of this lane's unit within a tile
  uint32_t col[KTl::kInstr];     // byte offset of the unit within its row
  uint32_t lds_base;             // wave-uniform LDS offset of this wavefront's first KB
  __device__ __forceinline__ KCopy(int wv, int lane) {
#pragma unroll
    for (int i = 0; i < KTl::kInstr; ++i) {
      const int e = (wv * KTl::kInstr + i) * kWave + lane;
      const int r = e / KTl::kUnits, p = e % KTl::kUnits;
      row[i] = (uint32_t)r;
      col[i] = (uint32_t)((p ^ (r % KTl::kUnits)) * 16);
    }
    lds_base = __builtin_amdgcn_readfirstlane((uint32_t)(wv * KTl::kInstr * kWave * 16));
  }
};

template <typename T, int D>
__device__ __forceinline__ void ktile_dma(const char* kb, int j0, int N, char* tile,
                                          const KCopy<T, D>& cp, bool real) {
  using KTl = KTile<T, D>;
  const int j0e = real ? j0 : 0;
  const uint32_t lim = (uint32_t)(N - 1 - j0e);     // last row of the sequence, tile-relative
  const char* base = kb + (int64_t)j0e * KTl::kRowBytes;
  const uint32_t lds = (uint32_t)(uintptr_t)(lds_ptr_t)tile + cp.lds_base;
#pragma unroll
  for (int i = 0; i < KTl::kInstr; ++i)
    dma16_sbase(base, min(cp.row[i], lim) * KTl::kRowBytes + cp.col[i], lds + i * kWave * 16);
}

// With S - 1 tiles always in flight (an S-stage ring), tile t has landed once at most
// S - 2 younger tiles (and whatever was issued after them) are outstanding; loads issued
// before it are complete too.
template <typename T, int D, int S>
__device__ __forceinline__ void ktile_wait() {
  asm_wait_vmcnt<(S - 2) * KTile<T, D>::kInstr>();
}

// Fragment of key row r (0..63 within the tile) for chunk step s and lane group g16.
template <typename T, int D>
__device__ __forceinline__ uint4 ktile_frag(const char* lds, int r, int s, int g16) {
  using KTl = KTile<T, D>;
  const int u = s * 4 + g16;
  return *reinterpret_cast<const uint4*>(lds + r * KTl::kRowBytes + ((u ^ (r % KTl::kUnits)) * 16));
}

// Row tiles of one row group (first tile tile0) as wavefront wv sees them:
//   slot i <  FT : tile tile0 + wv + 4 i, for every key of every K tile ("own" tiles);
//   slot FT + r  : tile tile0 + 4 FT + r, shared by the four wavefronts -- wavefront wv
//                  takes only the 16 keys of subtile wv of each 64-key K tile.
// With T tiles in the group, FT = T / 4 and RT = T % 4 give every wavefront the same
// number of (row tile, 16-key subtile) products, 4 FT + RT per K tile; the plain
// "tile w + 4i" ownership would leave three wavefronts computing a padding tile.
template <int FT>
__device__ __forceinline__ int slot_tile(int tile0, int wv, int i) {
  return i < FT ? tile0 + wv + 4 * i : tile0 + 4 * FT + (i - FT);
}

// Register loads before the K copies (query fragments, the colsum pass's row
// normalisers): from asm (untracked by the compiler, so an explicit vmcnt wait
// covers them and the K tiles keep streaming) when the wavefront holds at most
// kAsyncSlots slots; with more, register pressure makes the compiler copy values
// between registers before they can have landed, so those instances use ordinary loads
// and the compiler's own waits.
constexpr int kAsyncSlots = 6;
template <int NQ>
__device__ __forceinline__ u32x4_t slot_load16(const void* p) {
  if constexpr (NQ <= kAsyncSlots) return async_load16(p);
  else return __builtin_bit_cast(u32x4_t, load16(p));
}
template <int NQ>
__device__ __forceinline__ float slot_load4(const float* p) {
  if constexpr (NQ <= kAsyncSlots) return async_load4(p);
  else return *p;
}

// Query fragments of the wavefront's slots (slot_load16): valid only after the first
// tile wait and q_fence().  Padding rows (m >= M) read row M - 1; their logits are
// masked (stats) or weighted by 2^-inf (colsum).
template <typename T, int D, int FT, int NQ>
__device__ __forceinline__ void load_q_frags(const ScoreArgs& a, int h, int b, int tile0, int wv,
                                             int c16, int g16,
                                             u32x4_t (&qf)[NQ][RowChunks<T, D>::kSteps]) {
  constexpr int NS = RowChunks<T, D>::kSteps;
  const T* qb = reinterpret_cast<const T*>(a.q);
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int m = min(slot_tile<FT>(tile0, wv, i) * 16 + c16, a.M - 1);   // lane: row l % 16
    const int g = m / a.n_rows;
    const int r = m - g * a.n_rows;
    const T* row = qb + (int64_t)(h * a.G + g) * a.q_head_stride + (int64_t)(b * a.n_rows + r) * D;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[i][s] = slot_load16<NQ>(row + chunk_elem<T, D>(s, g16));
  }
}

// After the first tile wait: the slot registers may be read from here on.
template <int NQ, int NS>
__device__ __forceinline__ void q_fence(u32x4_t (&qf)[NQ][NS]) {
  if constexpr (NQ <= kAsyncSlots) {
#pragma unroll
    for (int i = 0; i < NQ; ++i)
#pragma unroll
      for (int s = 0; s < NS; ++s) reg_fence(qf[i][s]);
  } else {
    wait_vmcnt<0>();         // compiler-visible: no wait of its own inside the stream
  }
}

template <int NQ>
__device__ __forceinline__ void cr_fence(float (&cr)[NQ][4]) {
  if constexpr (NQ <= kAsyncSlots) {
#pragma unroll
    for (int i = 0; i < NQ; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) reg_fence(cr[i][t]);
  }
}

// Copies of tiles 0..S-2 of a chunk (dummies past its end).
template <typename T, int D, int S>
__device__ __forceinline__ void ktile_issue(const char* kb, int c0, int ntiles, int N,
                                            char (*buf)[KTile<T, D>::kBytes],
                                            const KCopy<T, D>& cp) {
#pragma unroll
  for (int t = 0; t < S - 1; ++t) ktile_dma<T, D>(kb, c0 + t * KT, N, buf[t], cp, t < ntiles);
}

// The copies, then the wait for tile 0: every load issued before the copies (query
// fragments) has landed too.
template <typename T, int D, int S>
__device__ __forceinline__ void ktile_prologue(const char* kb, int c0, int ntiles, int N,
                                               char (*buf)[KTile<T, D>::kBytes],
                                               const KCopy<T, D>& cp) {
  ktile_issue<T, D, S>(kb, c0, ntiles, N, buf, cp);
  ktile_wait<T, D, S>();
}

// consume(tile, j0, t) for the tiles t of [c0, c0 + ntiles * KT), ntiles >= 1, after
// the prologue.  Tile t lands in buffer t % S; S - 1 copies stay in flight (dummies
// past the chunk's end) and all of them have landed when this returns.  The barrier
// at the top of each iteration also waits for the wavefront's own LDS traffic, so
// whatever consume(t - 1) wrote to LDS is visible to every wavefront in consume(t).
template <typename T, int D, int S, typename F>
__device__ __forceinline__ void ktile_stream(const char* kb, int c0, int ntiles, int N,
                                             char (*buf)[KTile<T, D>::kBytes],
                                             const KCopy<T, D>& cp, F&& consume) {
  int t = 0;
  do {
    if (t > 0) ktile_wait<T, D, S>();
    lds_barrier();           // tile t landed everywhere; buffer (t - 1) % S free
    const int tn = t + S - 1;
    ktile_dma<T, D>(kb, c0 + tn * KT, N, buf[tn % S], cp, tn < ntiles);
    consume(buf[t % S], c0 + t * KT, t);
  } while (++t < ntiles);
  asm_wait_vmcnt<0>();       // no copy still writes into the buffers
}

// Subtiles of a 64-key tile whose products the stats pass issues together before their
// results are used (16 registers per own tile per subtile); the row sums take each
// group's logits in one rebase_lse_update (one overflow check per group).  The products of
// one group are independent of the exp2 work of the previous one, so the matrix cores
// and the vector ALUs overlap.
template <int FT>
constexpr int sub_group() { return FT <= 2 ? 4 : (FT <= 4 ? 2 : 1); }

// Wavefronts per SIMD the score kernels are compiled for: two (256 registers each, so
// two workgroups share a compute unit) while a wavefront holds at most 12 16-byte query
// chunks, owns at most two row tiles and shares at most two (every Llama-3-8B-shaped
// scoring geometry); larger row sets get the whole register file and one wavefront per
// SIMD instead of spilling.
template <typename T, int D, int FT, int RT>
constexpr int score_waves() {
  constexpr int NS = RowChunks<T, D>::kSteps;
  return (FT + RT) * NS <= 12 && FT < 3 && RT < 3 && NS <= 4 ? 2 : 1;
}
template <typename T, int D, int FT, int RT>
constexpr int stats_waves() { return score_waves<T, D, FT, RT>(); }
// The colsum pass at Llama-3-8B-like row counts (bf16, d = 128, at most two own and one
// shared tile per wavefront) also fits three wavefronts per SIMD (<= 168 registers) with a
// 3-stage ring; the stats pass at three spills.  Three are faster on launches of many
// rounds of workgroups (32 layers of a batch of 8 sequences of 16K-32K tokens: colsum
// 3.2 -> 2.9 ms) and slower on launches of one or two rounds (32 layers of one 16K
// sequence, 1280 workgroups: 2-4%, the last round then leaving compute units idle), so
// the launch picks the instance by its workgroup count (kColsumThreeWaveUnits).
template <typename T, int D, int FT, int RT>
constexpr int colsum_max_waves() {
  return std::is_same<T, bf16_t>::value && D == 128 && FT <= 2 && RT <= 1
             ? 3 : score_waves<T, D, FT, RT>();
}
constexpr int kColsumThreeWaveUnits = 4096;

// Depth of the K ring of a kernel compiled for W wavefronts per SIMD (W workgroups per
// compute unit share its 160 KB of LDS): 4 stages of 16 KB (3 tiles in flight) for up
// to two workgroups, 3 for three; tiles over 16 KB (fp32 rows of 128) get 2.
template <typename T, int D, int W>
constexpr int ring_stages() { return KTile<T, D>::kBytes > 16384 ? 2 : (W >= 3 ? 3 : 4); }

// Per-wavefront row state of the stats pass: lane (c16, g16) holds row c16 of each
// slot's tile and keys 4*g16..4*g16+3 of every 16-key subtile; (mref, srow) is the
// running (reference, sum of 2^(x - reference)) of those logits in the log2 domain, mref
// starting finite (see rebase_lse_update).
template <int NQ>
struct StatsRows {
  int pos[NQ];
  bool live[NQ];
  float mref[NQ], srow[NQ];
};

template <int FT, int NQ>
__device__ __forceinline__ void stats_rows_init(const ScoreArgs& a, int tile0, int wv, int c16,
                                                int p0, StatsRows<NQ>& st) {
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const int m = slot_tile<FT>(tile0, wv, i) * 16 + c16;
    st.live[i] = m < a.M;
    st.pos[i] = p0 + (st.live[i] ? m % a.n_rows : 0);
    st.mref[i] = kLazyRefInit;
    st.srow[i] = 0.0f;
  }
}

// Logit of key j for a row at position pos, -inf where it is masked.  MASK bodies run
// only on tiles that reach past the sequence or past the first scoring position.
__device__ __forceinline__ float stats_mask(float x, int j, bool live, int pos, int N) {
  return (live && j < N && j <= pos) ? x : -INFINITY;
}

// Running sums of one 64-key tile for the wavefront's slots (A = keys, B = query rows).
template <typename T, int D, int FT, int RT, bool MASK>
__device__ __forceinline__ void stats_tile_body(const ScoreArgs& a, const char* lds, int j0, int N,
                                                int wv, int c16, int g16,
                                                const u32x4_t (&qf)[FT + RT][RowChunks<T, D>::kSteps],
                                                StatsRows<FT + RT>& st) {
  constexpr int NS = RowChunks<T, D>::kSteps;
  constexpr int SG = sub_group<FT>();
  f32x4_t accr[RT > 0 ? RT : 1];
  if constexpr (RT > 0) {                  // shared tiles: subtile wv only
    uint4 kf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) kf[s] = ktile_frag<T, D>(lds, wv * 16 + c16, s, g16);
#pragma unroll
    for (int r = 0; r < RT; ++r) accr[r] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int r = 0; r < RT; ++r) accr[r] = mma_step(T{}, kf[s], as_uint4(qf[FT + r][s]), accr[r]);
  }
  if constexpr (FT > 0) {
#pragma unroll
    for (int sg = 0; sg < KT / 16; sg += SG) {
      f32x4_t acc[SG][FT];
#pragma unroll
      for (int u = 0; u < SG; ++u) {
        uint4 kf[NS];
#pragma unroll
        for (int s = 0; s < NS; ++s) kf[s] = ktile_frag<T, D>(lds, (sg + u) * 16 + c16, s, g16);
#pragma unroll
        for (int i = 0; i < FT; ++i) acc[u][i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
          for (int i = 0; i < FT; ++i) acc[u][i] = mma_step(T{}, kf[s], as_uint4(qf[i][s]), acc[u][i]);
      }
      float x[FT][4 * SG];
#pragma unroll
      for (int i = 0; i < FT; ++i)
#pragma unroll
        for (int u = 0; u < SG; ++u)
#pragma unroll
          for (int t = 0; t < 4; ++t) {
            x[i][4 * u + t] = acc[u][i][t];
            if constexpr (MASK)
              x[i][4 * u + t] = stats_mask(x[i][4 * u + t], j0 + (sg + u) * 16 + 4 * g16 + t,
                                           st.live[i], st.pos[i], N);
          }
      rebase_lse_update<FT, 4 * SG>(x, a.scale_log2, st.mref, st.srow);
    }
  }
  if constexpr (RT > 0) {
    float x[RT][4];
#pragma unroll
    for (int r = 0; r < RT; ++r)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        x[r][t] = accr[r][t];
        if constexpr (MASK)
          x[r][t] = stats_mask(x[r][t], j0 + wv * 16 + 4 * g16 + t, st.live[FT + r], st.pos[FT + r], N);
      }
    rebase_lse_update<RT, 4>(x, a.scale_log2, st.mref + FT, st.srow + FT);
  }
}

template <typename T, int D, int FT, int RT>
__device__ __forceinline__ void stats_tile(const ScoreArgs& a, const char* lds, int j0, int N,
                                           int p0, int wv, int c16, int g16,
                                           const u32x4_t (&qf)[FT + RT][RowChunks<T, D>::kSteps],
                                           StatsRows<FT + RT>& st) {
  // masking only where the tile reaches past the first scoring position: padding rows
  // (not live) elsewhere accumulate harmless sums that are never stored
  if (j0 + KT - 1 > p0) stats_tile_body<T, D, FT, RT, true>(a, lds, j0, N, wv, c16, g16, qf, st);
  else stats_tile_body<T, D, FT, RT, false>(a, lds, j0, N, wv, c16, g16, qf, st);
}

// Merge the four lane groups that hold the same row: every lane ends with its row's
// (reference, sum) over the keys the wavefront has seen.
template <int NQ>
__device__ __forceinline__ void stats_rows_merge(StatsRows<NQ>& st) {
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const float m = st.mref[i];
    float s = st.srow[i];
    const float mx = fmaxf(fmaxf(m, shfl_xor_f<16>(m)), fmaxf(shfl_xor_f<32>(m), shfl_xor_f<48>(m)));
    s *= rescale(m, mx);
    s += shfl_xor_f<16>(s);
    s += shfl_xor_f<32>(s);
    st.mref[i] = mx;
    st.srow[i] = s;
  }
}

// Column sums of one 64-key tile (A = query rows, B = keys): for subtile u, lane
// (c16, g16) holds rows 4*g16..4*g16+3 of each slot's tile for key u*16 + c16.  cr = log2
// normaliser of each row (+inf for padding rows, whose terms are then exactly 0).  The
// subtiles are independent straight-line code, so the products of one overlap the exp2
// work of the previous one.  Ends with lane group g16 of every wavefront writing the
// wavefront's sums of subtile g16 to redw[g16 * 16 + c16].  MASK: the tile reaches past
// the first scoring position; row (slot i, 4*g16 + t) then sits at position
// p0 + ((rb[i] + t) mod n_rows), rb[i] being the row index of (slot i, 4*g16) mod n_rows.
template <typename T, int D, int FT, int RT, bool MASK>
__device__ __forceinline__ void colsum_tile_body(const ScoreArgs& a, const char* lds, int j0,
                                                 int N, int p0, int wv, int c16, int g16,
                                                 const u32x4_t (&qf)[FT + RT][RowChunks<T, D>::kSteps],
                                                 const float (&cr)[FT + RT][4],
                                                 const int (&rb)[FT + RT], float* redw) {
  constexpr int NS = RowChunks<T, D>::kSteps;
  // key j visible to row (slot i, 4*g16 + t).  The row's position is derived here, in
  // the rare masked body (the empty asm keeps the compiler from hoisting the 4 (FT + RT)
  // positions out of the loop, where they would hold registers across every tile);
  // padding rows (cr = +inf) contribute 0 whatever this says.
  auto visible = [&](int i, int t, int j) {
    int r = rb[i];
    asm volatile("" : "+v"(r));
    r += t;
#pragma unroll
    for (int w = 0; w < 3; ++w) r -= r >= a.n_rows ? a.n_rows : 0;   // t <= 3 < 4 n_rows
    return j < N && j <= p0 + r;
  };
  float colp[4] = {0.f, 0.f, 0.f, 0.f};
  if constexpr (FT > 0) {
#pragma unroll
    for (int u = 0; u < KT / 16; ++u) {
      uint4 kf[NS];
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[s] = ktile_frag<T, D>(lds, u * 16 + c16, s, g16);
      f32x4_t acc[FT];
#pragma unroll
      for (int i = 0; i < FT; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int i = 0; i < FT; ++i) acc[i] = mma_step(T{}, as_uint4(qf[i][s]), kf[s], acc[i]);
      const int j = j0 + u * 16 + c16;
#pragma unroll
      for (int i = 0; i < FT; ++i) {
        float e[4];
#pragma unroll
        for (int t = 0; t < 4; ++t) {
          e[t] = fast_exp2(fmaf(acc[i][t], a.scale_log2, -cr[i][t]));
          if constexpr (MASK) e[t] = visible(i, t, j) ? e[t] : 0.0f;
        }
        colp[u] += (e[0] + e[1]) + (e[2] + e[3]);
      }
    }
  }
  if constexpr (RT > 0) {                  // shared tiles: this wavefront's subtile only
    uint4 kf[NS];
#pragma unroll
    for (int s = 0; s < NS; ++s) kf[s] = ktile_frag<T, D>(lds, wv * 16 + c16, s, g16);
    f32x4_t accr[RT];
#pragma unroll
    for (int r = 0; r < RT; ++r) accr[r] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int s = 0; s < NS; ++s)
#pragma unroll
      for (int r = 0; r < RT; ++r) accr[r] = mma_step(T{}, as_uint4(qf[FT + r][s]), kf[s], accr[r]);
    const int j = j0 + wv * 16 + c16;
    float cp = 0.0f;
#pragma unroll
    for (int r = 0; r < RT; ++r) {
      float e[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        e[t] = fast_exp2(fmaf(accr[r][t], a.scale_log2, -cr[FT + r][t]));
        if constexpr (MASK) e[t] = visible(FT + r, t, j) ? e[t] : 0.0f;
      }
      cp += (e[0] + e[1]) + (e[2] + e[3]);
    }
#pragma unroll
    for (int u = 0; u < 4; ++u) colp[u] += u == wv ? cp : 0.0f;
  }
  redw[g16 * 16 + c16] = reduce_scatter_lane_groups(colp);
}

// Column sums of the tile at j0 from the four wavefronts' partials (red[w][key]):
// lanes 0..15 of wavefront w store keys w*16..w*16+15.
__device__ __forceinline__ void colsum_flush(const ScoreArgs& a, const float (*red)[KT], int j0,
                                             int c1, int wv, int lane, float* out,
                                             bool accumulate) {
  const int key = wv * 16 + lane;
  if (lane < 16 && j0 + key < c1) {
    const float v = ((red[0][key] + red[1][key]) + (red[2][key] + red[3][key])) * a.inv_G;
    if (accumulate) out[j0 + key] += v;
    else out[j0 + key] = v;
  }
}

template <typename T, int D, int FT, int RT>
__device__ __forceinline__ void colsum_tile(const ScoreArgs& a, const char* lds, int j0, int N,
                                            int p0, int wv, int c16, int g16,
                                            const u32x4_t (&qf)[FT + RT][RowChunks<T, D>::kSteps],
                                            const float (&cr)[FT + RT][4],
                                            const int (&rb)[FT + RT], float* redw) {
  if (j0 + KT - 1 > p0)
    colsum_tile_body<T, D, FT, RT, true>(a, lds, j0, N, p0, wv, c16, g16, qf, cr, rb, redw);
  else
    colsum_tile_body<T, D, FT, RT, false>(a, lds, j0, N, p0, wv, c16, g16, qf, cr, rb, redw);
}

template <typename T, int D, int FT, int RT>
__global__ __launch_bounds__(kThreads, (stats_waves<T, D, FT, RT>())) void score_stats_kernel(ScoreArgs a) {
  using KTl = KTile<T, D>;
  constexpr int S = ring_stages<T, D, stats_waves<T, D, FT, RT>()>();
  constexpr int NS = RowChunks<T, D>::kSteps;
  constexpr int NQ = FT + RT;
  prefetch_args(a.q, a.k, a.n_chunks, a.n_kv_heads, a.batch, a.chunk_keys, a.p0_from_end,
                a.kv_head_stride, a.q_head_stride, a.M, a.n_rows, a.G, a.M_pad, a.groups,
                a.offs);
  const int units = a.n_chunks * a.n_kv_heads * a.batch;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int chunk = unit % a.n_chunks, h = (unit / a.n_chunks) % a.n_kv_heads,
            b = unit / (a.n_chunks * a.n_kv_heads);
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int c0 = chunk * a.chunk_keys;
  if (c0 >= N) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int p0 = N - a.p0_from_end;
  const int c1 = min(N, c0 + a.chunk_keys);
  const int ntiles = (c1 - c0 + KT - 1) / KT;
  const char* kb = reinterpret_cast<const char*>(a.k) +
                   ((int64_t)h * a.kv_head_stride + s0 * D) * Elem<T>::kBytes;
  float* part = a.partial + ((int64_t)(b * a.n_kv_heads + h) * a.n_chunks + chunk) * a.M_pad;
  __shared__ __attribute__((aligned(16))) char ldsbuf[S][KTl::kBytes];
  __shared__ float2 xch[4][(RT > 0 ? RT : 1) * 16];   // shared-tile partials per wavefront
  const KCopy<T, D> kcp(wv, lane);

  for (int grp = 0; grp < a.groups; ++grp) {
    const int tile0 = grp * 4 * FT;
    // query fragments first, then the K copies: the first tile wait covers both, and
    // later tiles keep landing while the first ones are on the matrix cores
    lds_barrier();                         // previous row group done with the buffers
    u32x4_t qf[NQ][NS];
    load_q_frags<T, D, FT, NQ>(a, h, b, tile0, wv, c16, g16, qf);
    ktile_prologue<T, D, S>(kb, c0, ntiles, N, ldsbuf, kcp);
    q_fence(qf);                           // landed with the first tile
    StatsRows<NQ> st;
    stats_rows_init<FT, NQ>(a, tile0, wv, c16, p0, st);
    ktile_stream<T, D, S>(kb, c0, ntiles, N, ldsbuf, kcp,
                       [&](const char* lds, int j0, int) {
                         stats_tile<T, D, FT, RT>(a, lds, j0, N, p0, wv, c16, g16, qf, st);
                       });
    stats_rows_merge<NQ>(st);
#pragma unroll
    for (int i = 0; i < FT; ++i) {
      const int row = slot_tile<FT>(tile0, wv, i) * 16 + c16;
      if (g16 == 0 && row < a.M) part[row] = st.mref[i] + __log2f(st.srow[i]);
    }
    if constexpr (RT > 0) {                // the four wavefronts' shares of each shared row
      if (g16 == 0)
#pragma unroll
        for (int r = 0; r < RT; ++r) xch[wv][r * 16 + c16] = make_float2(st.mref[FT + r], st.srow[FT + r]);
      lds_barrier();
      if (tid < RT * 16) {
        const int r = tid / 16, row = (tile0 + 4 * FT + r) * 16 + (tid % 16);
        float m = xch[0][tid].x;
#pragma unroll
        for (int w = 1; w < 4; ++w) m = fmaxf(m, xch[w][tid].x);
        float sum = 0.0f;
#pragma unroll
        for (int w = 0; w < 4; ++w) sum += xch[w][tid].y * rescale(xch[w][tid].x, m);
        if (row < a.M) part[row] = m + __log2f(sum);
      }
    }
  }
}

// Stats pass with one K stream per wavefront (bf16, d = 128, every row tile of the head
// in each wavefront's registers: at most 9 tiles, i.e. 144 rows).  The workgroup's chunk
// is split into four runs of 16-key subtiles, one per wavefront; each wavefront streams
// its run through a private 4-stage ring of 4 KB subtiles (global->LDS copies, the same
// swizzle as the 64-key tiles) with its own vmcnt waits and no workgroup barrier, and
// keeps (reference, sum) of its lane's row of every tile.  The four runs' sums merge once
// at the end, through LDS, into the same chunk partial the four-wavefront kernel writes.
// A barrier per 64-key tile couples the four wavefronts of that kernel: with random bf16
// operands the stats arithmetic then slows the K stream by a sixth (2.6-2.9 ms for 14 GB
// against 2.3 ms for private rings, same arithmetic per byte, measured on MI355X).
// Ring depth of both per-wavefront passes: 3 subtiles in flight per wavefront (measured
// on the stats pass: 4 stages 1-2% faster than 5 or 3).
constexpr int kWaveStages = 4;
constexpr int kSubKeys = 16;
// Only on walks of at least this many 64-key tiles: every wavefront loads all the row
// tiles' queries (36 KB at 9 tiles), which short walks do not amortise (one 4096-token
// layer, 3-tile walks: 21.5 -> 24.9 us).
constexpr int kWaveStatsMinTiles = 32;

// One wavefront's run of 16-key subtiles (bf16, d = 128) through its private S-stage
// ring: subtile t lands in buf[t % S]; nothing is copied past the run's last subtile, so
// the waits of the run's last S - 2 subtiles count fewer copies in flight (measured on
// MI355X: 0.5% faster than dummy copies that keep every wait count fixed).  Lane l
// copies 16-byte unit e = i*64 + l
// (row e / 16) to its linear LDS position, fetching the unit that belongs there under the
// XOR swizzle of the 64-key tiles; rows past the sequence read its last row.
template <int S>
struct WaveRun {
  using KTl = KTile<bf16_t, 128>;
  static constexpr int kSubBytes = kSubKeys * KTl::kRowBytes;
  static constexpr int kCopies = kSubBytes / (kWave * 16);     // 4 instructions per subtile
  const char* kb;
  char (*buf)[kSubBytes];
  int w0, nw, N;
  uint32_t off[kCopies];         // the unit's byte offset within a subtile (row * 256 + column)
  __device__ __forceinline__ WaveRun(const char* kb_, char (*buf_)[kSubBytes], int w0_, int nw_,
                                     int N_, int lane)
      : kb(kb_), buf(buf_), w0(w0_), nw(nw_), N(N_) {
#pragma unroll
    for (int i = 0; i < kCopies; ++i) {
      const int e = i * kWave + lane, r = e / KTl::kUnits, u = e % KTl::kUnits;
      off[i] = (uint32_t)(r * KTl::kRowBytes + (u ^ (r % KTl::kUnits)) * 16);
    }
  }
  __device__ __forceinline__ void issue(int t) const {
    if (t >= nw) return;                       // wave-uniform
    const int js = w0 + t * kSubKeys;
    const uint32_t lim = (uint32_t)(N - 1 - js);
    const char* base = kb + (int64_t)js * KTl::kRowBytes;
    const uint32_t lds = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)(lds_ptr_t)buf[t % S]);
#pragma unroll
    for (int i = 0; i < kCopies; ++i) {
      const uint32_t r = off[i] / KTl::kRowBytes;      // a shift
      dma16_sbase(base, off[i] - (r - min(r, lim)) * KTl::kRowBytes, lds + i * kWave * 16);
    }
  }
  // vmcnt wait that leaves the copies of `ahead` younger subtiles in flight (at most A)
  template <int A>
  __device__ __forceinline__ void wait_ahead(int ahead) const {
    if constexpr (A == 0) {
      asm_wait_vmcnt<0>();
    } else {
      if (ahead >= A) asm_wait_vmcnt<A * kCopies>();
      else wait_ahead<A - 1>(ahead);
    }
  }
  // subtile t landed (the copies of subtiles t+1 .. min(t + S - 2, nw - 1) may still be
  // in flight; those of 0..S-2 were waited for before t = 0), and this wavefront's reads
  // of the buffer that the next copy refills are done
  __device__ __forceinline__ void wait(int t) const {
    if (t > 0) wait_ahead<S - 2>(nw - 1 - t);
    wait_lgkmcnt0();
  }
};

template <int NQ>
__global__ __launch_bounds__(kThreads, 2) void score_stats_wave_kernel(ScoreArgs a) {
  using T = bf16_t;
  constexpr int D = 128;
  constexpr int NS = RowChunks<T, D>::kSteps;
  constexpr int S = kWaveStages;
  constexpr int kSubBytes = WaveRun<S>::kSubBytes;
  static_assert(NQ * kSubKeys * sizeof(float2) <= kSubBytes, "exchange exceeds a ring buffer");
  prefetch_args(a.q, a.k, a.n_chunks, a.n_kv_heads, a.batch, a.chunk_keys, a.p0_from_end,
                a.kv_head_stride, a.q_head_stride, a.M, a.n_rows, a.G, a.M_pad, a.offs);
  const int units = a.n_chunks * a.n_kv_heads * a.batch;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int chunk = unit % a.n_chunks, h = (unit / a.n_chunks) % a.n_kv_heads,
            b = unit / (a.n_chunks * a.n_kv_heads);
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int c0 = chunk * a.chunk_keys;
  if (c0 >= N) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform for the copies
  const int g16 = lane >> 4, c16 = lane & 15;
  const int p0 = N - a.p0_from_end;
  const int c1 = min(N, c0 + a.chunk_keys);
  const int nsub = (c1 - c0 + kSubKeys - 1) / kSubKeys;
  const int per = (nsub + 3) / 4;                        // subtiles per wavefront
  const int w0 = c0 + wv * per * kSubKeys;               // first key of this wavefront's run
  const int nw = max(0, min(per, nsub - wv * per));      // wave-uniform
  const char* kb = reinterpret_cast<const char*>(a.k) +
                   ((int64_t)h * a.kv_head_stride + s0 * D) * Elem<T>::kBytes;
  float* part = a.partial + ((int64_t)(b * a.n_kv_heads + h) * a.n_chunks + chunk) * a.M_pad;
  __shared__ __attribute__((aligned(16))) char ring[4][S][kSubBytes];
  char (*buf)[kSubBytes] = ring[wv];

  float mref[NQ], srow[NQ];
#pragma unroll
  for (int i = 0; i < NQ; ++i) { mref[i] = kLazyRefInit; srow[i] = 0.0f; }
  if (nw > 0) {
    const WaveRun<S> run(kb, buf, w0, nw, N, lane);
    u32x4_t qf[NQ][NS];
    load_q_frags<T, D, 0, NQ>(a, h, b, 0, wv, c16, g16, qf);   // slot i = row tile i
#pragma unroll
    for (int t = 0; t < S - 1; ++t) run.issue(t);
    q_fence(qf);                               // queries and the first subtiles landed
    for (int t = 0; t < nw; ++t) {
      run.wait(t);
      run.issue(t + S - 1);
      const char* lds = buf[t % S];
      const int j0 = w0 + t * kSubKeys;
      uint4 kf[NS];
#pragma unroll
      for (int s = 0; s < NS; ++s) kf[s] = ktile_frag<T, D>(lds, c16, s, g16);
      f32x4_t acc[NQ];
#pragma unroll
      for (int i = 0; i < NQ; ++i) acc[i] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int i = 0; i < NQ; ++i) acc[i] = mma_step(T{}, kf[s], as_uint4(qf[i][s]), acc[i]);
      float x[NQ][4];
      if (j0 + kSubKeys - 1 > p0) {            // reaches past the first scoring position
#pragma unroll
        for (int i = 0; i < NQ; ++i) {
          const int m = i * 16 + c16;
          const bool live = m < a.M;
          const int pos = p0 + (live ? m % a.n_rows : 0);
#pragma unroll
          for (int t2 = 0; t2 < 4; ++t2) x[i][t2] = stats_mask(acc[i][t2], j0 + 4 * g16 + t2, live, pos, N);
        }
      } else {
#pragma unroll
        for (int i = 0; i < NQ; ++i)
#pragma unroll
          for (int t2 = 0; t2 < 4; ++t2) x[i][t2] = acc[i][t2];
      }
      rebase_lse_update<NQ, 4>(x, a.scale_log2, mref, srow);
    }
    asm_wait_vmcnt<0>();                       // no copy still writes into the ring
  }
  // the four lane groups of each row, then the four wavefronts' runs (each wavefront
  // writes into its own first ring buffer, which no copy of any wavefront targets now)
  float2* xw = reinterpret_cast<float2*>(&ring[wv][0][0]);
#pragma unroll
  for (int i = 0; i < NQ; ++i) {
    const float m = mref[i];
    float sm = srow[i];
    const float mx = fmaxf(fmaxf(m, shfl_xor_f<16>(m)), fmaxf(shfl_xor_f<32>(m), shfl_xor_f<48>(m)));
    sm *= rescale(m, mx);
    sm += shfl_xor_f<16>(sm);
    sm += shfl_xor_f<32>(sm);
    if (g16 == 0) xw[i * 16 + c16] = make_float2(mx, sm);
  }
  lds_barrier();
  if (tid < a.M) {
    float m = -INFINITY;
#pragma unroll
    for (int w = 0; w < 4; ++w) m = fmaxf(m, reinterpret_cast<const float2*>(&ring[w][0][0])[tid].x);
    float sum = 0.0f;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
      const float2 v = reinterpret_cast<const float2*>(&ring[w][0][0])[tid];
      sum += v.y * rescale(v.x, m);
    }
    part[tid] = m + __log2f(sum);
  }
}

// Merging each query row's chunk partials (log2-sum-exps, -inf for a chunk whose keys
// are all masked for the row) into log2 of its normaliser, in one of two layouts:
// - score_reduce_rows_kernel, for at most kReduceBatch chunks (long chunks: the
//   layer-major c3/c4 launches): a lane per row, 64 consecutive rows of one (KV head,
//   sequence) per wavefront, every chunk's partials of those rows one coalesced
//   256-byte read, all in flight at once, merged in chunk order;
// - score_reduce_chunks_kernel, for more chunks (short launches of one layer): a
//   wavefront per row, a lane per chunk, merged by shuffles.
// Both write rowc and, when asked, the row's natural-log LSE.
constexpr int kReduceBatch = 8;

__device__ __forceinline__ void reduce_store(const ScoreArgs& a, int64_t base, int h, int b,
                                             int m, float c) {
  a.rowc[base * a.M_pad + m] = c;
  if (a.lse_out != nullptr) {          // query head h * G + g, row b * n_rows + r
    const int g = m / a.n_rows, r = m - g * a.n_rows;
    a.lse_out[(int64_t)(h * a.G + g) * a.batch * a.n_rows + b * a.n_rows + r] =
        c * 0.6931471805599453f;
  }
}

__global__ __launch_bounds__(64) void score_reduce_rows_kernel(ScoreArgs a) {
  const int m = blockIdx.x * 64 + (int)threadIdx.x;
  const int h = blockIdx.y, b = blockIdx.z;
  if (m >= a.M_pad) return;
  const int64_t base = (int64_t)(b * a.n_kv_heads + h);
  if (m >= a.M) {   // padding rows: 2^(x - inf) = 0
    a.rowc[base * a.M_pad + m] = INFINITY;
    return;
  }
  const int N = (int)(a.offs[b + 1] - a.offs[b]);
  const int nch = (N + a.chunk_keys - 1) / a.chunk_keys;   // <= kReduceBatch
  const float* src = a.partial + base * a.n_chunks * a.M_pad + m;
  float p[kReduceBatch];
#pragma unroll
  for (int u = 0; u < kReduceBatch; ++u) p[u] = u < nch ? src[(int64_t)u * a.M_pad] : -INFINITY;
  float mm = -INFINITY, ss = 0.0f;
#pragma unroll
  for (int u = 0; u < kReduceBatch; ++u) {
    const float mx = fmaxf(mm, p[u]);
    ss = ss * rescale(mm, mx) + (p[u] > -INFINITY ? fast_exp2(p[u] - mx) : 0.0f);
    mm = mx;
  }
  reduce_store(a, base, h, b, m, mm + __log2f(ss));
}

__global__ __launch_bounds__(256) void score_reduce_chunks_kernel(ScoreArgs a) {
  const int lane = threadIdx.x & 63;
  const int m = blockIdx.x * 4 + (threadIdx.x >> 6);
  const int h = blockIdx.y, b = blockIdx.z;
  if (m >= a.M_pad) return;
  const int64_t base = (int64_t)(b * a.n_kv_heads + h);
  if (m >= a.M) {   // padding rows: 2^(x - inf) = 0
    if (lane == 0) a.rowc[base * a.M_pad + m] = INFINITY;
    return;
  }
  const int N = (int)(a.offs[b + 1] - a.offs[b]);
  const int nch = (N + a.chunk_keys - 1) / a.chunk_keys;
  float mm = -INFINITY, ss = 0.0f;
  for (int ch = lane; ch < nch; ch += 64) {
    const float p = a.partial[(base * a.n_chunks + ch) * a.M_pad + m];
    const float mx = fmaxf(mm, p);
    ss = ss * rescale(mm, mx) + (p > -INFINITY ? fast_exp2(p - mx) : 0.0f);
    mm = mx;
  }
  float mx = mm;
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) mx = fmaxf(mx, __shfl_xor(mx, o, 64));
  ss *= rescale(mm, mx);
#pragma unroll
  for (int o = 1; o < 64; o <<= 1) ss += __shfl_xor(ss, o, 64);
  if (lane == 0) reduce_store(a, base, h, b, m, mx + __log2f(ss));
}

template <typename T, int D, int FT, int RT, int W>
__global__ __launch_bounds__(kThreads, W) void score_colsum_kernel(ScoreArgs a) {
  using KTl = KTile<T, D>;
  constexpr int S = ring_stages<T, D, W>();
  constexpr int NS = RowChunks<T, D>::kSteps;
  constexpr int NQ = FT + RT;
  prefetch_args(a.q, a.k, a.n_chunks, a.n_kv_heads, a.batch, a.chunk_keys, a.p0_from_end,
                a.kv_head_stride, a.q_head_stride, a.M, a.n_rows, a.G, a.M_pad, a.groups,
                a.offs);
  const int units = a.n_chunks * a.n_kv_heads * a.batch;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int chunk = unit % a.n_chunks, h = (unit / a.n_chunks) % a.n_kv_heads,
            b = unit / (a.n_chunks * a.n_kv_heads);
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int c0 = chunk * a.chunk_keys;
  if (c0 >= N) return;
  const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
  const int g16 = lane >> 4, c16 = lane & 15;
  const int p0 = N - a.p0_from_end;
  const int c1 = min(N, c0 + a.chunk_keys);
  const int ntiles = (c1 - c0 + KT - 1) / KT;
  const char* kb = reinterpret_cast<const char*>(a.k) +
                   ((int64_t)h * a.kv_head_stride + s0 * D) * Elem<T>::kBytes;
  const float* rowc = a.rowc + (int64_t)(b * a.n_kv_heads + h) * a.M_pad;
  // row normalisers: natural-log LSE supplied by the caller, or log2-domain rowc
  const float* lse_in = a.lse_in;
  const float cr_scale = lse_in != nullptr ? kLog2e : 1.0f;
  float* out = a.raw + (int64_t)h * a.total_rows + s0;
  __shared__ __attribute__((aligned(16))) char ldsbuf[S][KTl::kBytes];
  __shared__ float red[2][4][KT];          // per-wavefront column partials, double-buffered
  const KCopy<T, D> kcp(wv, lane);

  for (int grp = 0; grp < a.groups; ++grp) {
    const int tile0 = grp * 4 * FT;
    lds_barrier();                         // previous row group done with the buffers
    // query fragments and row normalisers first (asm loads, clamped rows), then the K
    // copies; the first tile wait covers all of them
    u32x4_t qf[NQ][NS];
    load_q_frags<T, D, FT, NQ>(a, h, b, tile0, wv, c16, g16, qf);
    float cr[NQ][4];
#pragma unroll
    for (int i = 0; i < NQ; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int m = min(slot_tile<FT>(tile0, wv, i) * 16 + 4 * g16 + t, a.M - 1);
        const int g = m / a.n_rows, r = m - g * a.n_rows;
        const float* src = lse_in != nullptr
                               ? lse_in + (int64_t)(h * a.G + g) * (a.q_head_stride / D) +
                                     b * a.n_rows + r
                               : rowc + m;
        cr[i][t] = slot_load4<NQ>(src);
      }
    ktile_prologue<T, D, S>(kb, c0, ntiles, N, ldsbuf, kcp);
    q_fence(qf);                           // landed with the first tile
    cr_fence<NQ>(cr);
#pragma unroll
    for (int i = 0; i < NQ; ++i)
#pragma unroll
      for (int t = 0; t < 4; ++t) {
        const int m = slot_tile<FT>(tile0, wv, i) * 16 + 4 * g16 + t;
        cr[i][t] = m < a.M ? cr[i][t] * cr_scale : INFINITY;   // padding rows add 0
      }
    int rb[NQ];
#pragma unroll
    for (int i = 0; i < NQ; ++i) rb[i] = min(slot_tile<FT>(tile0, wv, i) * 16 + 4 * g16, a.M - 1) % a.n_rows;
    int prev_j0 = c0;
    ktile_stream<T, D, S>(kb, c0, ntiles, N, ldsbuf, kcp,
                       [&](const char* lds, int j0, int t) {
                         // the previous tile's partials are visible after the stream's barrier
                         if (t > 0) colsum_flush(a, red[(t - 1) & 1], prev_j0, c1, wv, lane, out, grp > 0);
                         colsum_tile<T, D, FT, RT>(a, lds, j0, N, p0, wv, c16, g16, qf, cr, rb,
                                                   red[t & 1][wv]);
                         prev_j0 = j0;
                       });
    lds_barrier();
    colsum_flush(a, red[(ntiles - 1) & 1], prev_j0, c1, wv, lane, out, grp > 0);
  }
}

// Colsum pass with one K stream per wavefront, as the stats pass above (bf16, d = 128,
// at most 9 row tiles, long walks): each wavefront streams its run of 16-key subtiles
// through a private 4-stage ring, computes every row tile's products (A = query rows),
// sums each key's column in-lane (4 rows of each tile) and over the four lane groups, and
// writes the keys itself; no LDS reduction across wavefronts.  Row r's normaliser enters
// as the products' initial accumulator, -c_r / s (s = log2(e) / sqrt(d)), so that
// 2^(s acc) = 2^(s x - c_r) and the normalisers share the accumulator registers (next to
// the query fragments at two wavefronts per SIMD there is no room for them); they are
// staged once per workgroup in LDS and read as 16-byte broadcasts for every subtile.
template <int NQ>
__global__ __launch_bounds__(kThreads, 2) void score_colsum_wave_kernel(ScoreArgs a) {
  using T = bf16_t;
  constexpr int D = 128;
  constexpr int NS = RowChunks<T, D>::kSteps;
  constexpr int S = kWaveStages;
  constexpr int kSubBytes = WaveRun<S>::kSubBytes;
  prefetch_args(a.q, a.k, a.n_chunks, a.n_kv_heads, a.batch, a.chunk_keys, a.p0_from_end,
                a.kv_head_stride, a.q_head_stride, a.M, a.n_rows, a.G, a.M_pad, a.offs);
  const int units = a.n_chunks * a.n_kv_heads * a.batch;
  const int unit = xcd_unit(units);
  if (unit >= units) return;
  const int chunk = unit % a.n_chunks, h = (unit / a.n_chunks) % a.n_kv_heads,
            b = unit / (a.n_chunks * a.n_kv_heads);
  const int64_t s0 = a.offs[b];
  const int N = (int)(a.offs[b + 1] - s0);
  const int c0 = chunk * a.chunk_keys;
  if (c0 >= N) return;
  const int tid = threadIdx.x, lane = tid & 63;
  const int wv = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int g16 = lane >> 4, c16 = lane & 15;
  const int p0 = N - a.p0_from_end;
  const int c1 = min(N, c0 + a.chunk_keys);
  const int nsub = (c1 - c0 + kSubKeys - 1) / kSubKeys;
  const int per = (nsub + 3) / 4;
  const int w0 = c0 + wv * per * kSubKeys;
  const int nw = max(0, min(per, nsub - wv * per));
  const char* kb = reinterpret_cast<const char*>(a.k) +
                   ((int64_t)h * a.kv_head_stride + s0 * D) * Elem<T>::kBytes;
  float* out = a.raw + (int64_t)h * a.total_rows + s0;
  __shared__ __attribute__((aligned(16))) char ring[4][S][kSubBytes];
  __shared__ __attribute__((aligned(16))) float cinit[NQ * 16];
  // -c_r / s per row from the natural-log LSE of the caller or the log2-domain merged
  // partials; -inf for padding rows, whose terms are then exactly 0
  if (tid < NQ * 16) {
    float c = -INFINITY;
    if (tid < a.M) {
      float cr;
      if (a.lse_in != nullptr) {
        const int g = tid / a.n_rows, r = tid - g * a.n_rows;
        cr = a.lse_in[(int64_t)(h * a.G + g) * (a.q_head_stride / D) + b * a.n_rows + r] * kLog2e;
      } else {
        cr = a.rowc[(int64_t)(b * a.n_kv_heads + h) * a.M_pad + tid];
      }
      c = -cr / a.scale_log2;
    }
    cinit[tid] = c;
  }
  lds_barrier();
  if (nw == 0) return;                         // no barrier follows
  const WaveRun<S> run(kb, ring[wv], w0, nw, N, lane);
  u32x4_t qf[NQ][NS];
  load_q_frags<T, D, 0, NQ>(a, h, b, 0, wv, c16, g16, qf);
#pragma unroll
  for (int t = 0; t < S - 1; ++t) run.issue(t);
  q_fence(qf);
  for (int t = 0; t < nw; ++t) {
    run.wait(t);
    run.issue(t + S - 1);
    const char* lds = ring[wv][t % S];
    const int j0 = w0 + t * kSubKeys, j = j0 + c16;
    uint4 kf[NS];
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2) kf[s2] = ktile_frag<T, D>(lds, c16, s2, g16);
    // lane (c16, g16) accumulates rows 16 i + 4 g16 + t2 of tile i for key j, starting
    // from those rows' -c_r / s
    f32x4_t acc[NQ];
#pragma unroll
    for (int i = 0; i < NQ; ++i) {
      const float4 c = *reinterpret_cast<const float4*>(&cinit[i * 16 + 4 * g16]);
      acc[i] = f32x4_t{c.x, c.y, c.z, c.w};
    }
#pragma unroll
    for (int s2 = 0; s2 < NS; ++s2)
#pragma unroll
      for (int i = 0; i < NQ; ++i) acc[i] = mma_step(T{}, as_uint4(qf[i][s2]), kf[s2], acc[i]);
    float colp = 0.0f;
    if (j0 + kSubKeys - 1 > p0) {              // reaches past the first scoring position
      int mb = 4 * g16;                        // row positions derived here, not hoisted
      asm volatile("" : "+v"(mb));
#pragma unroll
      for (int i = 0; i < NQ; ++i) {
        float e[4];
#pragma unroll
        for (int t2 = 0; t2 < 4; ++t2) {
          const int m = i * 16 + mb + t2;
          const int r = m < a.M ? m % a.n_rows : 0;     // padding rows add 0 anyway
          e[t2] = fast_exp2(acc[i][t2] * a.scale_log2);
          e[t2] = (j < N && j <= p0 + r) ? e[t2] : 0.0f;
        }
        colp += (e[0] + e[1]) + (e[2] + e[3]);
      }
    } else {
#pragma unroll
      for (int i = 0; i < NQ; ++i)
        colp += (fast_exp2(acc[i][0] * a.scale_log2) + fast_exp2(acc[i][1] * a.scale_log2)) +
                (fast_exp2(acc[i][2] * a.scale_log2) + fast_exp2(acc[i][3] * a.scale_log2));
    }
    colp += shfl_xor_f<16>(colp);
    colp += shfl_xor_f<32>(colp);
    if (g16 == 0 && j < c1) out[j] = colp * a.inv_G;
  }
  asm_wait_vmcnt<0>();                         // no copy still writes into the ring
}

template <typename T, int D, int FT, int RT>
hipError_t launch_typed(const ScoreArgs& a, const dge_geom_t& g, hipStream_t st) {
  const dim3 grid(xcd_grid(a.n_chunks * g.n_kv_heads * g.batch));
  if (a.lse_in == nullptr) {   // normalisers computed here: stats and reduce first
    constexpr int NQW = 4 * FT + RT;         // row tiles of a single row group
    if constexpr (std::is_same<T, bf16_t>::value && D == 128 && (NQW == 8 || NQW == 9)) {
      if (a.groups == 1 && a.n_tiles == NQW && a.iters >= kWaveStatsMinTiles)
        hipLaunchKernelGGL((score_stats_wave_kernel<NQW>), grid, dim3(kThreads), 0, st, a);
      else
        hipLaunchKernelGGL((score_stats_kernel<T, D, FT, RT>), grid, dim3(kThreads), 0, st, a);
    } else {
      hipLaunchKernelGGL((score_stats_kernel<T, D, FT, RT>), grid, dim3(kThreads), 0, st, a);
    }
    if (a.n_chunks <= kReduceBatch)
      hipLaunchKernelGGL(score_reduce_rows_kernel, dim3((a.M_pad + 63) / 64, g.n_kv_heads, g.batch),
                         dim3(64), 0, st, a);
    else
      hipLaunchKernelGGL(score_reduce_chunks_kernel, dim3(a.M_pad / 4, g.n_kv_heads, g.batch),
                         dim3(256), 0, st, a);
  }
  // the colsum pass with its own split of the keys (it reads only the merged normalisers)
  ScoreArgs ac = a;
  ac.iters = a.c_iters;
  ac.chunk_keys = a.c_chunk_keys;
  ac.n_chunks = a.c_n_chunks;
  const int cunits = ac.n_chunks * g.n_kv_heads * g.batch;
  const dim3 gridc(xcd_grid(cunits));
  constexpr int W2 = score_waves<T, D, FT, RT>(), W3 = colsum_max_waves<T, D, FT, RT>();
  constexpr int NQC = 4 * FT + RT;
  if constexpr (std::is_same<T, bf16_t>::value && D == 128 && (NQC == 8 || NQC == 9)) {
    if (ac.groups == 1 && ac.n_tiles == NQC && ac.iters >= kWaveStatsMinTiles) {
      hipLaunchKernelGGL((score_colsum_wave_kernel<NQC>), gridc, dim3(kThreads), 0, st, ac);
      return hipGetLastError();
    }
  }
  if (W3 != W2 && cunits >= kColsumThreeWaveUnits)
    hipLaunchKernelGGL((score_colsum_kernel<T, D, FT, RT, W3>), gridc, dim3(kThreads), 0, st, ac);
  else
    hipLaunchKernelGGL((score_colsum_kernel<T, D, FT, RT, W2>), gridc, dim3(kThreads), 0, st, ac);
  return hipGetLastError();
}

// (FT, RT): own tiles per wavefront and shared tiles per row group.  Instantiated for
// RT = 0 with FT = 1..9, and for FT <= 3 with RT = 1..3, within the register budget of
// 36 16-byte query fragments per lane (FT + RT <= 36 / steps).
template <typename T, int D>
hipError_t launch_split(const ScoreArgs& a, const dge_geom_t& g, int ft, int rt, hipStream_t st) {
  constexpr int kSlots = 36 / RowChunks<T, D>::kSteps;
#define DGE_SPLIT(F, R)                                                  \
  if constexpr ((F) + (R) <= kSlots) {                                  \
    if (ft == (F) && rt == (R)) return launch_typed<T, D, F, R>(a, g, st); \
  }
  DGE_SPLIT(1, 0) DGE_SPLIT(2, 0) DGE_SPLIT(3, 0) DGE_SPLIT(4, 0) DGE_SPLIT(5, 0)
  DGE_SPLIT(6, 0) DGE_SPLIT(7, 0) DGE_SPLIT(8, 0) DGE_SPLIT(9, 0)
  DGE_SPLIT(0, 1) DGE_SPLIT(0, 2) DGE_SPLIT(0, 3)
  DGE_SPLIT(1, 1) DGE_SPLIT(1, 2) DGE_SPLIT(1, 3)
  DGE_SPLIT(2, 1) DGE_SPLIT(2, 2) DGE_SPLIT(2, 3)
  DGE_SPLIT(3, 1) DGE_SPLIT(3, 2) DGE_SPLIT(3, 3)
#undef DGE_SPLIT
  return hipErrorInvalidValue;
}

// Register budget for query fragments: tiles-per-wavefront * steps <= 36 16-byte chunks.
int max_mtw(const dge_geom_t& g) {
  const int steps = g.head_dim * (g.dtype == DGE_BF16 ? 2 : 4) / 64;
  const int m = 36 / steps;
  return m > 9 ? 9 : m;
}

}  // namespace

SeqOffsets seq_offsets(const dge_geom_t& g) {
  SeqOffsets o{};
  o.dev = g.kv_offsets;
  o.batch = g.batch;
  o.use_inline = g.batch <= kInlineSeqs && g.kv_offsets_host[g.batch] <= INT32_MAX;
  if (o.use_inline)
    for (int b = 0; b <= g.batch; ++b) o.inl[b] = (int32_t)g.kv_offsets_host[b];
  return o;
}

int64_t total_rows(const dge_geom_t& g) { return g.kv_offsets_host[g.batch]; }

int64_t max_seq_rows(const dge_geom_t& g) {
  int64_t m = 0;
  for (int b = 0; b < g.batch; ++b) {
    const int64_t n = g.kv_offsets_host[b + 1] - g.kv_offsets_host[b];
    m = n > m ? n : m;
  }
  return m;
}

ScorePlan plan_score(const dge_geom_t& g, int rows_mode) {
  ScorePlan p{};
  switch (rows_mode) {
    case DGE_ROWS_DRAFT: p.n_rows = g.k_draft; p.p0_from_end = g.k_draft; break;
    case DGE_ROWS_WINDOW: p.n_rows = g.window; p.p0_from_end = g.k_draft + g.window; break;
    default: p.n_rows = g.window + g.k_draft; p.p0_from_end = g.window + g.k_draft; break;
  }
  const int G = g.n_q_heads / g.n_kv_heads;
  p.M = G * p.n_rows;
  p.M_pad = (p.M + 15) / 16 * 16;
  p.n_tiles = p.M_pad / 16;
  const int cap = max_mtw(g);
  const int T = p.n_tiles, ft = T / 4, rt = T % 4;
  if (rt == 0 && ft <= cap) {              // every wavefront owns T / 4 tiles
    p.groups = 1; p.ft = ft; p.rt = 0;
  } else if (ft <= 3 && ft + rt <= cap) {  // own tiles + subtile-split shared tiles
    p.groups = 1; p.ft = ft; p.rt = rt;
  } else {                                 // row groups of 4 * ft tiles, padding in the last
    const int per_wave = (T + 3) / 4;
    p.groups = per_wave <= cap ? 1 : (per_wave + cap - 1) / cap;
    p.ft = (per_wave + p.groups - 1) / p.groups;
    p.rt = 0;
  }
  // Every workgroup loads its query fragments once and streams several 64-key tiles:
  // about one tile-walk per 256 tiles of the launch, at most 64 or 128 tiles (measured on
  // MI355X: one 4096-token layer of 8 KV heads 0.5 us faster with 3 tiles per workgroup
  // than with 2; 32 layers scored in one launch, at 16K tokens or at batch 8 of 16K-32K
  // tokens, 3% and 7% faster walking 64 tiles than 16).
  const int64_t tiles_total = (int64_t)g.n_kv_heads * ((total_rows(g) + KT - 1) / KT);
  const int64_t nmax = max_seq_rows(g);
  // The chunk count follows from that walk length; the chunks are then made equal (the
  // longest sequence's tiles spread evenly over its chunks instead of leaving a last
  // chunk of a few keys).  Walks may reach 128 tiles while a pass keeps at least
  // kLongWalkUnits workgroups (32 layers of a batch of 8 sequences of 16K-32K tokens:
  // 1.3% faster than at most 64; 32 layers of one 16K sequence, 768 workgroups at 128:
  // 1.5% slower, so it stays at 64).
  constexpr int64_t kLongWalkUnits = 4096;
  const int64_t seq_tiles = nmax > 0 ? (nmax + KT - 1) / KT : 1;
  auto balanced = [&](int walk) {
    auto even = [&](int cap) {
      const int w = walk < 1 ? 1 : (walk > cap ? cap : walk);
      const int64_t chunks = (seq_tiles + w - 1) / w;
      return (int)((seq_tiles + chunks - 1) / chunks);
    };
    const int w128 = even(128);
    const int64_t units128 = (seq_tiles + w128 - 1) / w128 * g.n_kv_heads * g.batch;
    return units128 >= kLongWalkUnits ? w128 : even(64);
  };
  int iters = balanced((int)((tiles_total + 255) / 256));
  p.tiles_per_wave = iters;
  p.chunk_keys = KT * iters;
  p.n_chunks = (int)((nmax + p.chunk_keys - 1) / p.chunk_keys);
  if (p.n_chunks < 1) p.n_chunks = 1;
  // the colsum pass walks about one tile per 512 of the launch (twice the workgroups of
  // the stats pass on small launches: one 4096-token layer of 8 KV heads 0.6 us faster
  // with 2 tiles per colsum workgroup and 3 per stats workgroup than with 3 and 3)
  const int citers = balanced((int)((tiles_total + 511) / 512));
  p.c_tiles = citers;
  p.c_chunk_keys = KT * citers;
  p.c_n_chunks = (int)((nmax + p.c_chunk_keys - 1) / p.c_chunk_keys);
  if (p.c_n_chunks < 1) p.c_n_chunks = 1;
  return p;
}

size_t score_workspace_bytes(const dge_geom_t& g, const ScorePlan& p) {
  const size_t units = (size_t)g.batch * g.n_kv_heads;
  return units * p.n_chunks * p.M_pad * sizeof(float) + units * p.M_pad * sizeof(float) + 256;
}

hipError_t launch_score(const dge_geom_t& g, const ScorePlan& p, const void* q, const void* k,
                        const float* row_lse, float* raw, void* ws, hipStream_t st,
                        float* lse_out) {
  ScoreArgs a{};
  a.lse_in = row_lse;
  a.lse_out = lse_out;
  a.q = q;
  a.k = k;
  a.raw = raw;
  const size_t units = (size_t)g.batch * g.n_kv_heads;
  a.partial = reinterpret_cast<float*>(ws);
  a.rowc = ws == nullptr ? nullptr : a.partial + units * p.n_chunks * p.M_pad;
  a.offs = seq_offsets(g);
  a.kv_head_stride = g.kv_head_stride;
  a.q_head_stride = (int64_t)g.batch * p.n_rows * g.head_dim;
  a.total_rows = total_rows(g);
  a.n_kv_heads = g.n_kv_heads;
  a.batch = g.batch;
  a.G = g.n_q_heads / g.n_kv_heads;
  a.n_rows = p.n_rows;
  a.p0_from_end = p.p0_from_end;
  a.M = p.M;
  a.M_pad = p.M_pad;
  a.n_tiles = p.n_tiles;
  a.groups = p.groups;
  a.iters = p.tiles_per_wave;
  a.chunk_keys = p.chunk_keys;
  a.n_chunks = p.n_chunks;
  a.c_iters = p.c_tiles;
  a.c_chunk_keys = p.c_chunk_keys;
  a.c_n_chunks = p.c_n_chunks;
  a.scale_log2 = kLog2e / sqrtf((float)g.head_dim);
  a.inv_G = 1.0f / (float)a.G;
  if (g.dtype == DGE_BF16) {
    return g.head_dim == 128 ? launch_split<bf16_t, 128>(a, g, p.ft, p.rt, st)
                             : launch_split<bf16_t, 64>(a, g, p.ft, p.rt, st);
  }
  return g.head_dim == 128 ? launch_split<float, 128>(a, g, p.ft, p.rt, st)
                           : launch_split<float, 64>(a, g, p.ft, p.rt, st);
}

}  // namespace dge
