// Host-side launch interface between the C ABI (api.hip) and the kernel files.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dge.h"

namespace dge {

// How dge_score splits one layer over the GPU.  Derived from the geometry alone so
// that dge_workspace_size and dge_score always agree.
struct ScorePlan {
  int n_rows;          // scoring rows per sequence
  int p0_from_end;     // first scoring position = N_b - p0_from_end
  int M;               // G * n_rows query rows per KV head and sequence
  int M_pad;           // M rounded up to 16
  int n_tiles;         // 16-row tiles (M_pad / 16)
  int ft;              // row tiles each wavefront owns in a row group (all keys)
  int rt;              // shared row tiles, split across wavefronts by key subtile
  int groups;          // row groups of 4 * ft + rt tiles covering all tiles
  int tiles_per_wave;  // 64-key iterations per workgroup (stats pass)
  int chunk_keys;      // keys per workgroup (4 wavefronts)
  int n_chunks;        // workgroups per (sequence, KV head)
  int c_tiles;         // the same three for the colsum pass, which only needs the merged
  int c_chunk_keys;    // row normalisers and may split the keys differently
  int c_n_chunks;
};

struct SeqOffsets;
SeqOffsets seq_offsets(const dge_geom_t& g);
int64_t total_rows(const dge_geom_t& g);
int64_t max_seq_rows(const dge_geom_t& g);
ScorePlan plan_score(const dge_geom_t& g, int rows_mode);
size_t score_workspace_bytes(const dge_geom_t& g, const ScorePlan& p);

hipError_t launch_score(const dge_geom_t& g, const ScorePlan& p, const void* q, const void* k,
                        const float* row_lse, float* raw, void* ws, hipStream_t stream,
                        float* lse_out = nullptr);

size_t select_workspace_bytes(const dge_geom_t& g);
hipError_t launch_select_topb(const dge_geom_t& g, const float* scores, int pool_kernel,
                              int n_tail, int n_select, int32_t* idx, int32_t* n_kept, void* ws,
                              hipStream_t stream);
hipError_t launch_select_compact(const dge_geom_t& g, const float* scores, int pool_kernel,
                                 int n_tail, int n_select, int32_t* idx, int32_t* n_kept,
                                 const void* k, const void* v, void* k_out, void* v_out, void* ws,
                                 hipStream_t stream);
hipError_t launch_select_compact_layers(const dge_geom_t& g, int n_layers, const float* scores,
                                        int pool_kernel, int n_tail, const int32_t* n_select_host,
                                        int32_t* idx, int32_t* n_kept, const void* k, const void* v,
                                        void* k_out, void* v_out, void* ws, hipStream_t stream);
hipError_t launch_select_streaming(const dge_geom_t& g, int n_sink, int n_recent, int32_t* idx,
                                   int32_t* n_kept, hipStream_t stream);

hipError_t launch_compact(const dge_geom_t& g, const int32_t* idx, const int32_t* n_kept,
                          int n_select, int n_tail, const void* k, const void* v, void* k_out,
                          void* v_out, hipStream_t stream);
hipError_t launch_compact_inplace(const dge_geom_t& g, const int32_t* idx, const int32_t* n_kept,
                                  int n_select, int n_tail, void* k, void* v, hipStream_t stream);

hipError_t launch_rope(int n_heads, int n_rows, int head_dim, int dtype, int64_t head_stride,
                       const int32_t* positions, double theta, void* x, hipStream_t stream);

size_t project_workspace_bytes(int n_rows, int hidden, int n_heads, int head_dim);
hipError_t launch_project_rope(int n_rows, int hidden, const void* x, int n_heads, int head_dim,
                               const void* w, const int32_t* positions, double theta, void* out,
                               void* ws, hipStream_t stream);

int cache_attention_max_group();
hipError_t launch_cache_attention(const dge_geom_t& g, const void* q, int n_q, int q_from_end,
                                  const void* k_c, const void* v_c, int n_select, int n_tail,
                                  const int32_t* n_kept, float* out, float* lse,
                                  hipStream_t stream);

hipError_t launch_evicted_mass(const dge_geom_t& g, const void* q, int n_q, int q_from_end,
                               const void* k_c, int n_select, int n_tail, const int32_t* n_kept,
                               const float* lse_full, float* rho, float* beta, float* l_match,
                               hipStream_t stream);

hipError_t launch_retained_runs(const dge_geom_t& g, const int32_t* idx, const int32_t* n_kept,
                                int n_select, int32_t* runs, float* mean_len, hipStream_t stream);

size_t h2o_workspace_bytes(const dge_geom_t& g);
hipError_t launch_h2o(const dge_geom_t& g, const void* q_all, const void* k, const float* lse,
                      float* colsum, void* ws, hipStream_t stream);

}  // namespace dge
