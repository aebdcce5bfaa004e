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
constexpr int kWaves = 4;             // waves per unit (a workgroup, or half of one)
constexpr int kMinSplitPages = 16;    // smallest page range a split workgroup gets
constexpr int kMinRangePagesMany = 256;  // ... in bf16 launches of at least a round of units
constexpr int kMaxPagesTwoUnit = 2048;  // longest units run two per workgroup (bf16, unsplit)
constexpr int kMaxLaunchRoutes = 65535;  // routes per launch and KV heads: grid dimension limits
constexpr int kOrderBuckets = 64;        // range-size classes of the dispatch order
constexpr int64_t kMaxOrderItems = int64_t(1) << 20;  // largest split launch given a dispatch order

struct AppendArgs {
  void* k_pool;
  void* v_pool;
  float* k_scale;  // fp8 pools: [num_pages][Hkv]
  float* v_scale;
  const uint16_t* k_new;
  const uint16_t* v_new;
  kf_route* routes;
  const int32_t* tail_route;
  const int32_t* page_ids;
  int32_t* err_flags;
  int32_t num_seqs, num_kv_heads, num_routes, num_pages, num_page_ids;
  int32_t head_major;  // pools [Hkv][num_pages][...] instead of [num_pages][Hkv][...]
};

struct PartialArgs {
  const uint16_t* q;
  const void* k_pool;
  const void* v_pool;
  const float* k_scale;
  const float* v_scale;
  const kf_route* routes;
  const int32_t* route_list;  // routes to process (NULL: all, in order)
  const int32_t* page_ids;
  float* o_part;
  float* lse_part;
  float* ws_ml;         // [launched routes * Hkv * max_chunks][G][2] (max, sum); chunked units only
  float* ws_o;          // [launched routes * Hkv * max_chunks][G][kDim]
  int32_t* err_flags;
  int32_t num_seqs, num_q_heads, num_kv_heads, group;
  int32_t num_routes, max_pages_per_route;
  int32_t num_units_routes;  // routes launched: num_list, or num_routes without a list
  int32_t chunk_pages, max_chunks;  // a unit of n pages uses ceil(n / chunk_pages) workgroups
  int32_t units_per_wg;  // 2: unsplit bf16 launch, two units per 512-thread workgroup
  // Split launches of several rounds: the dispatch order of the work items,
  // written by order_kernel before the partial kernel runs (NULL: grid
  // order).  [0] the item count, [1] unused, then per item (launch position
  // u, KV head << 16 | range index).
  uint32_t* order;
  int32_t head_major;    // pools [Hkv][num_pages][...] instead of [num_pages][Hkv][...]
  int32_t num_pages, num_page_ids;
  float scale_log2;     // scale * log2(e): scores are kept in the base-2 domain
  // Fused tail append (kf_decode_step; all NULL otherwise): the route that is
  // its sequence's tail takes the step's token into its pages and attends
  // over it; routes[].tok_end is advanced by the merge kernel.
  const uint16_t* k_new;       // [num_seqs][Hkv][kDim]
  const uint16_t* v_new;
  const int32_t* tail_route;   // [num_seqs]
  void* k_pool_w;              // the pools, writable
  void* v_pool_w;
  float* k_scale_w;            // fp8 pools: the scales, writable
  float* v_scale_w;
};

struct MergeArgs {
  const float* o_part;
  const float* lse_part;
  const int32_t* seq_route_begin;
  float* out;
  float* lse_out;
  int32_t* err_flags;
  int32_t num_seqs, num_routes, num_q_heads;
  // Tail bookkeeping of a fused step (tail_route NULL: none): for each
  // sequence whose tail took the step's token, tok_end += 1; the append's
  // error flags are raised here.
  kf_route* routes;
  const int32_t* tail_route;
  const int32_t* page_ids;
  int32_t num_pages, num_page_ids;
};

struct WorkspaceLayout {
  size_t ml_off, o_off, order_off, total;  // order_off: 0 without a dispatch order
};

// How the pages of each (route, KV head) unit are spread over workgroups.
// One workgroup owns a whole unit when the units fill whole rounds of the
// GPU's resident workgroups (two per compute unit), or, with equal routes,
// when they spread evenly over the compute units (units mod CUs is 0 or at
// least 3/4 of the CUs); otherwise units are cut into chunks of chunk_pages
// pages, so the dispatcher balances them, and a combine kernel follows:
// other equal units take the fewest chunks giving at least two work items
// per CU, spread evenly so; other launches about 12 chunks per resident slot (6 for
// fp8) when units outnumber slots,
// else about one (four when the page table shows ragged routes), an odd
// number of chunks for the longest unit where it matters.
struct ChunkPlan {
  int32_t chunk_pages, max_chunks;
};
// True when the page table holds under 90% of num_routes * max_pages_per_route
// entries: the routes reserve different page counts (ragged lengths).
bool ragged_table(int64_t num_page_ids, int32_t num_routes, int32_t max_pages_per_route);
// Ranges per resident slot when units outnumber slots (12 bf16, 6 fp8); from
// that many units per slot on, every unit runs whole.
int64_t ranges_per_slot(bool fp8);
// listed: a launch over a route list (kf_partial_attn_subset), whose routes
// the page table's reading does not describe; the equal-unit rules are
// skipped for it.
ChunkPlan plan_chunks(int32_t num_routes, int32_t num_kv_heads, int32_t max_pages_per_route,
                      bool ragged, bool fp8, bool listed);
// Units per workgroup of a partial-attention launch of num_launch routes
// (1 or 2); route_list: a launch over a route list (kf_partial_attn_subset).
int32_t units_per_workgroup(bool fp8, bool route_list, const ChunkPlan& plan, int32_t num_launch,
                            int32_t num_kv_heads, int32_t max_pages_per_route);
// A split launch of at least two rounds of the GPU's `slots` resident
// workgroups (and at most kMaxOrderItems work items) runs its work items
// in a computed order, largest ranges first (order_kernel).
bool ordered_dispatch(const ChunkPlan& plan, int32_t num_launch, int32_t num_kv_heads,
                      int64_t slots);
WorkspaceLayout workspace_layout(int32_t num_routes, int32_t num_kv_heads, int32_t group,
                                 int32_t max_chunks, bool ordered);

// Address of the current device's scratch array (KF_SCRATCH_BYTES, for
// kf_decode_step_no_alloc), looked up once per device.
hipError_t scratch_address(void** out);

hipError_t launch_append(const AppendArgs& a, bool fp8, hipStream_t stream);
hipError_t launch_partial(const PartialArgs& a, bool fp8, hipStream_t stream);
hipError_t launch_merge(const MergeArgs& a, hipStream_t stream);
hipError_t launch_gather(const PartialArgs& a, bool fp8, int route, int max_tokens, void* out_k,
                         void* out_v, hipStream_t stream);

}  // namespace kf
