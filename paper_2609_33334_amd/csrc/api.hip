// C ABI of the eviction-step library: argument validation on the host, then
// asynchronous launches on the caller's stream.  Nothing is launched when a
// check fails.  See include/dge.h for the contract of every entry point.
#include <cstddef>
#include <cstdint>
#include <mutex>

#include "dge.h"
#include "dge_internal.hpp"

using dge::ScorePlan;

namespace {

// bound on row counts (sequence lengths, n_select), so that n_select + n_tail and the
// kernels' row indices stay within int32
constexpr int32_t kMaxRows = INT32_MAX / 2;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

dge_status_t check_geom(const dge_geom_t* g) {
  if (g == nullptr) return DGE_ERR_INVALID;
  if (g->batch < 1 || g->n_kv_heads < 1 || g->n_q_heads < 1) return DGE_ERR_INVALID;
  if (g->n_q_heads % g->n_kv_heads != 0) return DGE_ERR_INVALID;
  if (g->n_q_heads / g->n_kv_heads > 64) return DGE_ERR_UNSUPPORTED;
  if (g->window < 0 || g->k_draft < 0) return DGE_ERR_INVALID;
  if (g->dtype != DGE_BF16 && g->dtype != DGE_F32) return DGE_ERR_INVALID;
  if (g->head_dim != 64 && g->head_dim != 128) return DGE_ERR_UNSUPPORTED;
  if (g->kv_offsets == nullptr || g->kv_offsets_host == nullptr) return DGE_ERR_INVALID;
  if ((reinterpret_cast<uintptr_t>(g->kv_offsets) & 7u) != 0) return DGE_ERR_INVALID;
  const int64_t* o = g->kv_offsets_host;
  if (o[0] != 0) return DGE_ERR_INVALID;
  for (int b = 0; b < g->batch; ++b) {
    if (o[b + 1] < o[b]) return DGE_ERR_INVALID;
    if (o[b + 1] - o[b] > (int64_t)INT32_MAX / 2) return DGE_ERR_UNSUPPORTED;
  }
  if (g->kv_head_stride < o[g->batch] * (int64_t)g->head_dim) return DGE_ERR_INVALID;
  if ((g->kv_head_stride * (g->dtype == DGE_BF16 ? 2 : 4)) % 16 != 0) return DGE_ERR_INVALID;
  return DGE_OK;
}

int64_t seq_rows(const dge_geom_t* g, int b) {
  return g->kv_offsets_host[b + 1] - g->kv_offsets_host[b];
}

dge_status_t check_tail(const dge_geom_t* g, int32_t n_tail) {
  if (n_tail < 0) return DGE_ERR_INVALID;
  for (int b = 0; b < g->batch; ++b)
    if (seq_rows(g, b) < n_tail) return DGE_ERR_INVALID;
  return DGE_OK;
}

dge_status_t hip_status(hipError_t e) { return e == hipSuccess ? DGE_OK : DGE_ERR_HIP; }

// Scratch of dge_score_noalloc: one fixed array per GPU, held until the process ends.  In
// host code `scratch` names a host-side stand-in, never the device memory; the device
// address is resolved once per device with that device current and kept in scratch_ptr.
static __device__ __align__(256) unsigned char scratch[DGE_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxDevices = 64;
std::mutex scratch_mu;
void* scratch_ptr[kMaxDevices];

dge_status_t scratch_of_current_device(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return DGE_ERR_HIP;
  std::lock_guard<std::mutex> lock(scratch_mu);
  if (scratch_ptr[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr)
      return DGE_ERR_HIP;
    scratch_ptr[dev] = p;
  }
  *out = scratch_ptr[dev];
  return DGE_OK;
}

// Checks shared by dge_score and dge_score_noalloc (everything but the workspace).
dge_status_t check_score(const dge_geom_t* geom, int32_t rows, const void* q, const void* k,
                         const float* raw) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (rows < DGE_ROWS_WINDOW_DRAFT || rows > DGE_ROWS_WINDOW) return DGE_ERR_INVALID;
  if (!q || !k || !raw || !aligned16(q) || !aligned16(k) || !aligned16(raw)) return DGE_ERR_INVALID;
  for (int b = 0; b < geom->batch; ++b)
    if (seq_rows(geom, b) < (int64_t)geom->window + geom->k_draft || seq_rows(geom, b) < 1)
      return DGE_ERR_INVALID;
  if (dge::plan_score(*geom, rows).n_rows <= 0) return DGE_ERR_INVALID;
  return DGE_OK;
}

}  // namespace

extern "C" {

int dge_abi_version(void) { return DGE_ABI_VERSION; }

const char* dge_status_string(int status) {
  switch (status) {
    case DGE_OK: return "DGE_OK";
    case DGE_ERR_INVALID: return "DGE_ERR_INVALID: argument violates the contract";
    case DGE_ERR_UNSUPPORTED: return "DGE_ERR_UNSUPPORTED: valid request not implemented by this build";
    case DGE_ERR_WORKSPACE: return "DGE_ERR_WORKSPACE: workspace missing or too small";
    case DGE_ERR_HIP: return "DGE_ERR_HIP: HIP launch or runtime failure";
    default: return "unknown dge status";
  }
}

dge_status_t dge_workspace_size(const dge_geom_t* geom, int32_t op, size_t* bytes) {
  if (bytes == nullptr) return DGE_ERR_INVALID;
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  switch (op) {
    case DGE_OP_SCORE: {
      // the largest scoring-row set (window + draft) bounds every mode
      const ScorePlan p = dge::plan_score(*geom, DGE_ROWS_WINDOW_DRAFT);
      size_t best = dge::score_workspace_bytes(*geom, p);
      for (int m = 1; m <= 2; ++m) {
        const size_t s = dge::score_workspace_bytes(*geom, dge::plan_score(*geom, m));
        best = s > best ? s : best;
      }
      *bytes = best;
      return DGE_OK;
    }
    case DGE_OP_SELECT: *bytes = dge::select_workspace_bytes(*geom); return DGE_OK;
    case DGE_OP_H2O: *bytes = dge::h2o_workspace_bytes(*geom); return DGE_OK;
    default: return DGE_ERR_INVALID;
  }
}

dge_status_t dge_score(const dge_geom_t* geom, int32_t rows, const void* q, const void* k,
                       float* raw, void* ws, size_t ws_bytes, hipStream_t stream) {
  dge_status_t st = check_score(geom, rows, q, k, raw);
  if (st != DGE_OK) return st;
  const ScorePlan p = dge::plan_score(*geom, rows);
  if (ws == nullptr || !aligned16(ws) || ws_bytes < dge::score_workspace_bytes(*geom, p))
    return DGE_ERR_WORKSPACE;
  return hip_status(dge::launch_score(*geom, p, q, k, nullptr, raw, ws, stream));
}

dge_status_t dge_score_with_lse(const dge_geom_t* geom, int32_t rows, const void* q,
                                const void* k, float* raw, float* row_lse, void* ws,
                                size_t ws_bytes, hipStream_t stream) {
  dge_status_t st = check_score(geom, rows, q, k, raw);
  if (st != DGE_OK) return st;
  if (row_lse == nullptr || !aligned16(row_lse)) return DGE_ERR_INVALID;
  const ScorePlan p = dge::plan_score(*geom, rows);
  if (ws == nullptr || !aligned16(ws) || ws_bytes < dge::score_workspace_bytes(*geom, p))
    return DGE_ERR_WORKSPACE;
  return hip_status(dge::launch_score(*geom, p, q, k, nullptr, raw, ws, stream, row_lse));
}

dge_status_t dge_score_noalloc(const dge_geom_t* geom, int32_t rows, const void* q,
                               const void* k, float* raw, hipStream_t stream) {
  dge_status_t st = check_score(geom, rows, q, k, raw);
  if (st != DGE_OK) return st;
  const ScorePlan p = dge::plan_score(*geom, rows);
  if (dge::score_workspace_bytes(*geom, p) > DGE_NOALLOC_SCRATCH_BYTES) return DGE_ERR_WORKSPACE;
  void* ws = nullptr;
  if ((st = scratch_of_current_device(&ws)) != DGE_OK) return st;
  return hip_status(dge::launch_score(*geom, p, q, k, nullptr, raw, ws, stream));
}

dge_status_t dge_score_lse(const dge_geom_t* geom, int32_t rows, const void* q, const void* k,
                           const float* row_lse, float* raw, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (rows < DGE_ROWS_WINDOW_DRAFT || rows > DGE_ROWS_WINDOW) return DGE_ERR_INVALID;
  if (!q || !k || !raw || !row_lse || !aligned16(q) || !aligned16(k) || !aligned16(raw) ||
      !aligned16(row_lse))
    return DGE_ERR_INVALID;
  for (int b = 0; b < geom->batch; ++b)
    if (seq_rows(geom, b) < (int64_t)geom->window + geom->k_draft || seq_rows(geom, b) < 1)
      return DGE_ERR_INVALID;
  const ScorePlan p = dge::plan_score(*geom, rows);
  if (p.n_rows <= 0) return DGE_ERR_INVALID;
  if (p.groups != 1) return DGE_ERR_UNSUPPORTED;
  return hip_status(dge::launch_score(*geom, p, q, k, row_lse, raw, nullptr, stream));
}

dge_status_t dge_select_topb(const dge_geom_t* geom, const float* scores, int32_t pool_kernel,
                             int32_t n_tail, int32_t n_select, int32_t* idx, int32_t* n_kept,
                             void* ws, size_t ws_bytes, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (pool_kernel < 1 || (pool_kernel & 1) == 0) return DGE_ERR_INVALID;
  if (n_select < 0 || n_select > kMaxRows) return DGE_ERR_INVALID;
  if ((st = check_tail(geom, n_tail)) != DGE_OK) return st;
  if (!scores || !n_kept || (n_select > 0 && !idx) || !aligned16(scores) || !aligned16(idx) ||
      !aligned16(n_kept))
    return DGE_ERR_INVALID;
  if (ws == nullptr || !aligned16(ws) || ws_bytes < dge::select_workspace_bytes(*geom))
    return DGE_ERR_WORKSPACE;
  return hip_status(
      dge::launch_select_topb(*geom, scores, pool_kernel, n_tail, n_select, idx, n_kept, ws, stream));
}

dge_status_t dge_select_compact(const dge_geom_t* geom, const float* scores, int32_t pool_kernel,
                                int32_t n_tail, int32_t n_select, int32_t* idx, int32_t* n_kept,
                                const void* k, const void* v, void* k_out, void* v_out, void* ws,
                                size_t ws_bytes, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (pool_kernel < 1 || (pool_kernel & 1) == 0) return DGE_ERR_INVALID;
  if (n_select < 0 || n_select > kMaxRows) return DGE_ERR_INVALID;
  if ((st = check_tail(geom, n_tail)) != DGE_OK) return st;
  if (!scores || !n_kept || (n_select > 0 && !idx) || !aligned16(scores) || !aligned16(idx) ||
      !aligned16(n_kept))
    return DGE_ERR_INVALID;
  if (!k || !v || !k_out || !v_out || !aligned16(k) || !aligned16(v) || !aligned16(k_out) ||
      !aligned16(v_out))
    return DGE_ERR_INVALID;
  if (ws == nullptr || !aligned16(ws) || ws_bytes < dge::select_workspace_bytes(*geom))
    return DGE_ERR_WORKSPACE;
  return hip_status(dge::launch_select_compact(*geom, scores, pool_kernel, n_tail, n_select, idx,
                                               n_kept, k, v, k_out, v_out, ws, stream));
}

dge_status_t dge_select_compact_layers(const dge_geom_t* geom, int32_t n_layers,
                                       const float* scores, int32_t pool_kernel, int32_t n_tail,
                                       const int32_t* n_select_host, int32_t* idx, int32_t* n_kept,
                                       const void* k, const void* v, void* k_out, void* v_out,
                                       void* ws, size_t ws_bytes, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (n_layers < 1 || !n_select_host) return DGE_ERR_INVALID;
  if (pool_kernel < 1 || (pool_kernel & 1) == 0) return DGE_ERR_INVALID;
  bool any_sel = false;
  for (int l = 0; l < n_layers; ++l) {
    if (n_select_host[l] < 0 || n_select_host[l] > kMaxRows) return DGE_ERR_INVALID;
    any_sel = any_sel || n_select_host[l] > 0;
  }
  if ((st = check_tail(geom, n_tail)) != DGE_OK) return st;
  if (!scores || !n_kept || (any_sel && !idx) || !aligned16(scores) || !aligned16(idx) ||
      !aligned16(n_kept))
    return DGE_ERR_INVALID;
  if (!k || !v || !k_out || !v_out || !aligned16(k) || !aligned16(v) || !aligned16(k_out) ||
      !aligned16(v_out))
    return DGE_ERR_INVALID;
  if (ws == nullptr || !aligned16(ws) || ws_bytes < dge::select_workspace_bytes(*geom))
    return DGE_ERR_WORKSPACE;
  return hip_status(dge::launch_select_compact_layers(*geom, n_layers, scores, pool_kernel, n_tail,
                                                      n_select_host, idx, n_kept, k, v, k_out,
                                                      v_out, ws, stream));
}

dge_status_t dge_select_streaming(const dge_geom_t* geom, int32_t n_sink, int32_t n_recent,
                                  int32_t* idx, int32_t* n_kept, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (n_sink < 0) return DGE_ERR_INVALID;
  if ((st = check_tail(geom, n_recent)) != DGE_OK) return st;
  if (!n_kept || !aligned16(n_kept) || (n_sink > 0 && (!idx || !aligned16(idx))))
    return DGE_ERR_INVALID;
  return hip_status(dge::launch_select_streaming(*geom, n_sink, n_recent, idx, n_kept, stream));
}

dge_status_t dge_compact(const dge_geom_t* geom, const int32_t* idx, const int32_t* n_kept,
                         int32_t n_select, int32_t n_tail, const void* k, const void* v,
                         void* k_out, void* v_out, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (n_select < 0 || n_select > kMaxRows) return DGE_ERR_INVALID;
  if ((st = check_tail(geom, n_tail)) != DGE_OK) return st;
  if (!n_kept || !k || !v || !k_out || !v_out || (n_select > 0 && !idx)) return DGE_ERR_INVALID;
  if (!aligned16(k) || !aligned16(v) || !aligned16(k_out) || !aligned16(v_out) ||
      !aligned16(n_kept) || (idx && !aligned16(idx)))
    return DGE_ERR_INVALID;
  return hip_status(
      dge::launch_compact(*geom, idx, n_kept, n_select, n_tail, k, v, k_out, v_out, stream));
}

dge_status_t dge_compact_inplace(const dge_geom_t* geom, const int32_t* idx,
                                 const int32_t* n_kept, int32_t n_select, int32_t n_tail, void* k,
                                 void* v, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (n_select < 0 || n_select > kMaxRows) return DGE_ERR_INVALID;
  if ((st = check_tail(geom, n_tail)) != DGE_OK) return st;
  if (!n_kept || !k || !v || (n_select > 0 && !idx) || k == v) return DGE_ERR_INVALID;
  if (!aligned16(k) || !aligned16(v) || !aligned16(n_kept) || (idx && !aligned16(idx)))
    return DGE_ERR_INVALID;
  return hip_status(dge::launch_compact_inplace(*geom, idx, n_kept, n_select, n_tail, k, v, stream));
}

dge_status_t dge_rope(int32_t n_heads, int32_t n_rows, int32_t head_dim, int32_t dtype,
                      int64_t head_stride, const int32_t* positions, double theta, void* x,
                      hipStream_t stream) {
  if (n_heads < 1 || n_rows < 0 || n_rows > kMaxRows) return DGE_ERR_INVALID;
  if (head_dim < 4 || head_dim > 128 || (head_dim & 3)) return DGE_ERR_UNSUPPORTED;
  if (dtype != DGE_BF16 && dtype != DGE_F32) return DGE_ERR_INVALID;
  if (!(theta > 1.0) || !(theta < 1e300)) return DGE_ERR_INVALID;
  if (head_stride < (int64_t)n_rows * head_dim) return DGE_ERR_INVALID;
  if ((head_stride * (dtype == DGE_BF16 ? 2 : 4)) % 8 != 0) return DGE_ERR_INVALID;  // 8-byte aligned heads
  if (n_rows > 0 && (!positions || !x)) return DGE_ERR_INVALID;
  if ((reinterpret_cast<uintptr_t>(positions) & 3) || !aligned16(x)) return DGE_ERR_INVALID;
  return hip_status(
      dge::launch_rope(n_heads, n_rows, head_dim, dtype, head_stride, positions, theta, x, stream));
}

static dge_status_t check_project(int32_t n_rows, int32_t hidden, int32_t n_heads,
                                  int32_t head_dim) {
  if (n_rows < 0 || n_heads < 1 || hidden < 1) return DGE_ERR_INVALID;
  if (head_dim != 64 && head_dim != 128) return DGE_ERR_UNSUPPORTED;
  if (hidden % 128 != 0) return DGE_ERR_UNSUPPORTED;
  if (n_rows > 64 * 65535 || (int64_t)n_heads * (head_dim / 16) > INT32_MAX / 16) return DGE_ERR_UNSUPPORTED;
  return DGE_OK;
}

dge_status_t dge_project_rope_workspace(int32_t n_rows, int32_t hidden, int32_t n_heads,
                                        int32_t head_dim, size_t* bytes) {
  if (bytes == nullptr) return DGE_ERR_INVALID;
  const dge_status_t st = check_project(n_rows, hidden, n_heads, head_dim);
  if (st != DGE_OK) return st;
  *bytes = dge::project_workspace_bytes(n_rows, hidden, n_heads, head_dim);
  return DGE_OK;
}

dge_status_t dge_project_rope(int32_t n_rows, int32_t hidden, const void* x, int32_t n_heads,
                              int32_t head_dim, const void* w, const int32_t* positions,
                              double theta, void* out, void* ws, size_t ws_bytes,
                              hipStream_t stream) {
  dge_status_t st = check_project(n_rows, hidden, n_heads, head_dim);
  if (st != DGE_OK) return st;
  if (!(theta > 1.0) || !(theta < 1e300)) return DGE_ERR_INVALID;
  if (n_rows == 0) return DGE_OK;
  if (!x || !w || !positions || !out || !aligned16(x) || !aligned16(w) || !aligned16(out) ||
      (reinterpret_cast<uintptr_t>(positions) & 3))
    return DGE_ERR_INVALID;
  const size_t need = dge::project_workspace_bytes(n_rows, hidden, n_heads, head_dim);
  if (need > 0 && (ws == nullptr || !aligned16(ws) || ws_bytes < need)) return DGE_ERR_WORKSPACE;
  return hip_status(dge::launch_project_rope(n_rows, hidden, x, n_heads, head_dim, w, positions,
                                             theta, out, ws, stream));
}

dge_status_t dge_cache_attention(const dge_geom_t* geom, const void* q, int32_t n_q,
                                 int32_t q_from_end, const void* k_c, const void* v_c,
                                 int32_t n_select, int32_t n_tail, const int32_t* n_kept,
                                 float* out, float* lse, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (n_q < 1 || n_select < 0 || n_select > kMaxRows || n_tail < 0 || q_from_end > n_tail ||
      n_select + n_tail < 1)
    return DGE_ERR_INVALID;
  if (!q || !k_c || !v_c || !n_kept || !out || !lse || !aligned16(q) || !aligned16(k_c) ||
      !aligned16(v_c) || !aligned16(out) || (reinterpret_cast<uintptr_t>(n_kept) & 3) ||
      (reinterpret_cast<uintptr_t>(lse) & 3))
    return DGE_ERR_INVALID;
  if (geom->n_q_heads / geom->n_kv_heads > dge::cache_attention_max_group())
    return DGE_ERR_UNSUPPORTED;
  return hip_status(dge::launch_cache_attention(*geom, q, n_q, q_from_end, k_c, v_c, n_select,
                                                n_tail, n_kept, out, lse, stream));
}

dge_status_t dge_evicted_mass(const dge_geom_t* geom, const void* q, int32_t n_q,
                              int32_t q_from_end, const void* k_c, int32_t n_select,
                              int32_t n_tail, const int32_t* n_kept, const float* lse_full,
                              float* rho, float* beta, float* l_match, hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (n_q < 1 || n_select < 0 || n_select > kMaxRows || n_tail < 1 || q_from_end > n_tail ||
      q_from_end < n_q)
    return DGE_ERR_INVALID;
  if (!q || !k_c || !n_kept || !lse_full || !rho || !beta || !l_match || !aligned16(q) ||
      !aligned16(k_c) || (reinterpret_cast<uintptr_t>(n_kept) & 3) ||
      (reinterpret_cast<uintptr_t>(lse_full) & 3) || (reinterpret_cast<uintptr_t>(rho) & 3) ||
      (reinterpret_cast<uintptr_t>(beta) & 3) || (reinterpret_cast<uintptr_t>(l_match) & 3))
    return DGE_ERR_INVALID;
  if (geom->n_q_heads / geom->n_kv_heads > dge::cache_attention_max_group())
    return DGE_ERR_UNSUPPORTED;
  return hip_status(dge::launch_evicted_mass(*geom, q, n_q, q_from_end, k_c, n_select, n_tail,
                                             n_kept, lse_full, rho, beta, l_match, stream));
}

dge_status_t dge_retained_runs(const dge_geom_t* geom, const int32_t* idx, const int32_t* n_kept,
                               int32_t n_select, int32_t* runs, float* mean_len,
                               hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (n_select < 0 || n_select > kMaxRows || !n_kept || !runs || !mean_len || (n_select > 0 && !idx))
    return DGE_ERR_INVALID;
  if ((reinterpret_cast<uintptr_t>(idx) & 3) || (reinterpret_cast<uintptr_t>(n_kept) & 3) ||
      (reinterpret_cast<uintptr_t>(runs) & 3) || (reinterpret_cast<uintptr_t>(mean_len) & 3))
    return DGE_ERR_INVALID;
  return hip_status(dge::launch_retained_runs(*geom, idx, n_kept, n_select, runs, mean_len, stream));
}

dge_status_t dge_h2o_colsum(const dge_geom_t* geom, const void* q_all, const void* k,
                            const float* lse, float* colsum, void* ws, size_t ws_bytes,
                            hipStream_t stream) {
  dge_status_t st = check_geom(geom);
  if (st != DGE_OK) return st;
  if (geom->dtype != DGE_BF16 || geom->head_dim != 128) return DGE_ERR_UNSUPPORTED;
  if (!q_all || !k || !colsum || !aligned16(q_all) || !aligned16(k) || !aligned16(colsum) ||
      (lse && !aligned16(lse)))
    return DGE_ERR_INVALID;
  if (lse == nullptr && geom->n_q_heads / geom->n_kv_heads > 4) return DGE_ERR_UNSUPPORTED;
  if (ws == nullptr || !aligned16(ws) || ws_bytes < dge::h2o_workspace_bytes(*geom))
    return DGE_ERR_WORKSPACE;
  return hip_status(dge::launch_h2o(*geom, q_all, k, lse, colsum, ws, stream));
}

dge_status_t dge_pyramid_budgets(int32_t B, int32_t w, int32_t n_layers, int32_t beta,
                                 int32_t* out_host) {
  if (out_host == nullptr || n_layers < 1 || beta < 1 || w < 0 || B < w) return DGE_ERR_INVALID;
  const int64_t c = (int64_t)B - w;
  const int64_t top = 2 * c - c / beta;
  const int64_t bottom = c / beta;
  const int64_t steps = n_layers > 1 ? (top - bottom) / (n_layers - 1) : 0;
  for (int l = 0; l < n_layers; ++l) out_host[l] = (int32_t)(top - l * steps + w);
  return DGE_OK;
}

}  // extern "C"
