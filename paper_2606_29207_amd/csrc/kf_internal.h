// Internal interface between the C-ABI layer (kf_api.cpp) and the gfx950
// kernels (kf_kernels.hip).  Not installed; callers use include/kf.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "kf.h"

namespace kf {

// Work decomposition of the partial-attention kernel, shared with workspace
// sizing on the host.
constexpr int kPage = KF_PAGE_SIZE;   // tokens per page
constexpr int kDim = KF_HEAD_DIM;     // head dimension
constexpr int kTilePages = 4;         // pages per wave tile (one lane group per page)
constexpr int kWaves = 4;             // waves per workgroup
constexpr int kChunkPages = 64;       // upper bound on pages per workgroup

struct AppendArgs {
  void* k_pool;
  void* v_pool;
  const uint16_t* k_new;
  const uint16_t* v_new;
  kf_route* routes;
  const int32_t* tail_route;
  const int32_t* page_ids;
  int32_t* err_flags;
  int32_t num_seqs, num_kv_heads, num_routes, num_pages, num_page_ids;
};

struct PartialArgs {
  const uint16_t* q;
  const void* k_pool;
  const void* v_pool;
  const float* k_scale;
  const float* v_scale;
  const kf_route* routes;
  const int32_t* page_ids;
  float* o_part;
  float* lse_part;
  int32_t* counters;    // [num_routes * Hkv], zero between calls
  float* ws_ml;         // [num_routes * Hkv * max_chunks][G][2] (max, sum)
  float* ws_o;          // [num_routes * Hkv * max_chunks][G][kDim]
  int32_t* err_flags;
  int32_t num_seqs, num_q_heads, num_kv_heads, group;
  int32_t num_routes, max_pages_per_route, max_chunks;
  int32_t num_pages, num_page_ids;
  float scale_log2;     // scale * log2(e): scores are kept in the base-2 domain
};

struct MergeArgs {
  const float* o_part;
  const float* lse_part;
  const int32_t* seq_route_begin;
  float* out;
  float* lse_out;
  int32_t* err_flags;
  int32_t num_seqs, num_routes, num_q_heads;
};

struct WorkspaceLayout {
  size_t counters_off, ml_off, o_off, total;
};

WorkspaceLayout workspace_layout(int32_t num_routes, int32_t num_kv_heads, int32_t group,
                                 int32_t max_chunks);
inline int32_t max_chunks_for(int32_t max_pages_per_route) {
  int32_t c = (max_pages_per_route + kChunkPages - 1) / kChunkPages;
  return c < 1 ? 1 : c;
}

hipError_t launch_append(const AppendArgs& a, hipStream_t stream);
hipError_t launch_partial(const PartialArgs& a, bool fp8, hipStream_t stream);
hipError_t launch_merge(const MergeArgs& a, hipStream_t stream);

}  // namespace kf
