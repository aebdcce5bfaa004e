// C-ABI layer of libkf: host-side argument checks, workspace sizing and
// kernel launches on the caller's stream.  Declarations and the contract of
// every entry point are in include/kf.h.
#include <math.h>
#include <stdint.h>

#include <atomic>
#include <initializer_list>

#include "kf.h"
#include "kf_internal.h"

namespace {

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// Checks shared by append and partial attention.
int check_shape(const kf_shape* s) {
  if (!s) return KF_ERR_INVALID_ARG;
  if (s->num_seqs < 0 || s->num_q_heads <= 0 || s->num_kv_heads <= 0 || s->num_pages < 1 ||
      s->num_page_ids < 0)
    return KF_ERR_INVALID_ARG;
  if (s->num_q_heads % s->num_kv_heads != 0) return KF_ERR_INVALID_ARG;
  if (s->num_q_heads / s->num_kv_heads > KF_MAX_GROUP) return KF_ERR_UNSUPPORTED;
  if (s->head_dim != KF_HEAD_DIM || s->page_size != KF_PAGE_SIZE) return KF_ERR_UNSUPPORTED;
  if (s->kv_dtype != KF_KV_BF16 && s->kv_dtype != KF_KV_FP8_E4M3) return KF_ERR_UNSUPPORTED;
  if (s->kv_layout != KF_KV_PAGE_MAJOR && s->kv_layout != KF_KV_HEAD_MAJOR) return KF_ERR_UNSUPPORTED;
  if (!isfinite(s->scale)) return KF_ERR_INVALID_ARG;
  // element offsets of the pools are formed in 64 bits; the grid needs
  // num_kv_heads <= 65535 (checked per call together with num_routes)
  return KF_OK;
}

hipStream_t as_stream(void* s) { return static_cast<hipStream_t>(s); }

}  // namespace

namespace kf {

namespace {
constexpr int kMaxDevices = 64;
std::atomic<int> g_cu_count[kMaxDevices];

// Compute units of the current device (queried once per device; 256 when no
// device is visible, so that sizes can be computed on a host without a GPU).
int cu_count() {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    (void)hipGetLastError();
    return 256;
  }
  int n = g_cu_count[dev].load(std::memory_order_relaxed);
  if (n > 0) return n;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) {
    (void)hipGetLastError();
    n = 256;
  }
  g_cu_count[dev].store(n, std::memory_order_relaxed);
  return n;
}
}  // namespace

bool ragged_table(int64_t num_page_ids, int32_t num_routes, int32_t max_pages_per_route) {
  // The page table is under 90% of routes x max pages: the routes reserve
  // different page counts.  reserved <= 2^62; ids * 10 < 2^35.
  const int64_t reserved = (int64_t)(num_routes > 0 ? num_routes : 0) *
                           (int64_t)(max_pages_per_route > 0 ? max_pages_per_route : 0);
  if (reserved <= 0) return false;
  const int64_t ids = num_page_ids > 0 ? num_page_ids : 0;
  // ids * 10 < reserved * 9, without forming reserved * 9 where it would
  // overflow (there ids * 10 < 2^35 is far below it)
  return reserved > INT64_MAX / 16 ? true : ids * 10 < reserved * 9;
}

int64_t ranges_per_slot(bool fp8) { return fp8 ? 6 : 12; }

namespace {
// plan_chunks for a GPU with `slots` resident workgroups (two per CU).
ChunkPlan plan_for_slots(int32_t num_routes, int32_t num_kv_heads, int32_t max_pages_per_route,
                         bool ragged, bool fp8, int64_t slots, bool listed) {
  const int64_t units = (int64_t)num_routes * num_kv_heads;
  const int32_t whole = max_pages_per_route > 0 ? max_pages_per_route : 1;
  if (units <= 0 || max_pages_per_route <= kMinSplitPages) return {whole, 1};
  // Whole units suit equal lengths only: a ragged batch that fills whole
  // rounds would wait for its longest unit, so it is cut into ranges like
  // any other.
  if (units >= slots && units % slots == 0 && !ragged) return {whole, 1};
  // The rules for equal units below trust the page table's reading, which
  // says nothing about the routes of a list (a part of a table), so
  // route-list launches skip them.
  // Equal units that do not fill whole rounds still stay whole when they
  // spread evenly over the compute units: every CU holds the same number of
  // units, or all but at most a quarter of the CUs hold one more (units mod
  // CUs is 0 or at least 3/4 of the CUs).  A CU streams about as fast with
  // one workgroup as with two, so the launch takes as long as its busiest
  // CU.  Measured against ranges on one box (units of 512 bf16 or 1024 fp8
  // pages): bf16 192 units -14%, 448 -10%, 704 -6%, 768 -3%, 960 -5%; fp8
  // 256 -11%, 448 -8%, 704 -5%, 768 -9%, 960 -6%.  Where a quarter to a half
  // of the CUs would hold one unit more (320, 384, 576, 832 units) whole
  // units were 3-15% slower than ranges.
  const int64_t cus = slots / 2;
  if (!ragged && !listed && units * 4 >= cus * 3) {
    const int64_t rem = units % cus;
    if (rem == 0 || rem * 4 >= cus * 3) return {whole, 1};
  }
  // Fewer units than slots: units of equal length run best as about one
  // range per slot, one round of workgroups; ragged routes need more ranges
  // for the dispatcher to balance.  More units than slots: about 12 ranges
  // per slot, 6 for fp8 pools, whose pages hold half the bytes, so that a
  // workgroup streams about as much either way.  From `many` ranges per slot
  // worth of units on, every unit is one range.
  const int64_t many = ranges_per_slot(fp8);
  if (units >= many * slots) return {whole, 1};
  // Other equal units: the fewest ranges per unit (2 to 16, of at least
  // kMinSplitPages pages) that give at least two work items per CU spread
  // evenly over the CUs (items mod CUs is 0 or at least 3/4 of the CUs).
  // Against the slot-count rule below (one box, units of 512 bf16 or 1024
  // fp8 pages): bf16 96 units -16%, 160 -9%, 320 -9%, 416 -11%; fp8 96 -16%,
  // 160 -2%, 320 -6%, 576 -2%, 640 -3%, 832 -1%; nowhere more than 0.9%
  // slower.
  if (!ragged && !listed) {
    for (int64_t m = 2; m <= 16; ++m) {
      const int64_t c = (max_pages_per_route + m - 1) / m;
      if (c < kMinSplitPages) break;
      if ((max_pages_per_route + c - 1) / c != m || units * m < 2 * cus) continue;
      const int64_t rem = units * m % cus;
      if (rem == 0 || rem * 4 >= cus * 3) return {(int32_t)c, (int32_t)m};
    }
  }
  const int64_t target = (units < slots ? (ragged ? 4 : 1) : many) * slots;
  int64_t c = (units * max_pages_per_route + target - 1) / target;  // < 2^31 * 2^15
  if (c < kMinSplitPages) c = kMinSplitPages;
  // With at least a round of bf16 units, ranges of fewer than
  // kMinRangePagesMany pages cost more in each workgroup's start and finish
  // than they gain in balance (960 units of 256 pages: 40-page ranges 331 us,
  // whole units 307 us; 512 ragged units: 94-page ranges 630 us, 205-page
  // ranges 605 us).  fp8 launches measured no gain from such a floor.
  if (!fp8 && units >= slots && c < kMinRangePagesMany) c = kMinRangePagesMany;
  if (c >= max_pages_per_route) return {whole, 1};
  int64_t m = (max_pages_per_route + c - 1) / c;
  // Workgroups are dealt round-robin over the 8 XCDs in launch order, chunk
  // index fastest, so with an even chunk count the chunk index alone picks
  // the XCD half (a multiple of 8: the XCD), and the units shorter than the
  // longest, whose high chunk indices are empty, leave those XCDs idle.  An
  // odd count rotates every chunk index over all XCDs.
  if ((units >= slots || ragged) && m % 2 == 0) {
    c = (max_pages_per_route + m) / (m + 1);
    if (c < kMinSplitPages) c = kMinSplitPages;
    m = (max_pages_per_route + c - 1) / c;
    // with many ranges the rounding can keep the count even: shorten the
    // ranges until it is odd (or the 16-page floor is reached); a bounded
    // search, so that planning stays O(1)
    for (int64_t cc = c - 1, tries = 0; m % 2 == 0 && cc >= kMinSplitPages && tries < 64;
         --cc, ++tries) {
      const int64_t mm = (max_pages_per_route + cc - 1) / cc;
      if (mm % 2 == 1) {
        c = cc;
        m = mm;
      }
    }
  }
  if (m > 65535) {
    m = 65535;
    c = (max_pages_per_route + m - 1) / m;
  }
  return {(int32_t)c, (int32_t)m};
}
}  // namespace

ChunkPlan plan_chunks(int32_t num_routes, int32_t num_kv_heads, int32_t max_pages_per_route,
                      bool ragged, bool fp8, bool listed) {
  return plan_for_slots(num_routes, num_kv_heads, max_pages_per_route, ragged, fp8,
                        2 * (int64_t)cu_count(), listed);
}

// Unsplit bf16 launches over the whole table with at least two units per
// CU, none longer than kMaxPagesTwoUnit pages, run two units per 512-thread
// workgroup, one workgroup per CU.  Both units of a CU then start at once:
// with 256-thread workgroups the second workgroup of each CU started ~3 us
// after the first, and the Llama layer ran 1.2-1.4% slower.  Units of 16384
// pages ran 1.1% slower in this mode.  Pairs go to CUs whole, so the busiest
// CU holds 2 * ceil(units / (2 * CUs)) units against ceil(units / CUs) with
// one unit per workgroup: units of more than 16 pages are paired only when
// ceil(units / CUs) is even (768 units of 512 pages: 538 us paired against
// 470 us single; 1280 units: 845 against 786).  Launches over a route list
// keep one unit per workgroup: they are made to run beside another launch,
// and a 512-thread workgroup needs the registers of a whole CU, so it waits
// until the other launch has left one entirely (the agentic query-first
// step took 1402 us this way against 1257 us).
int32_t units_per_workgroup(bool fp8, bool route_list, const ChunkPlan& plan, int32_t num_launch,
                            int32_t num_kv_heads, int32_t max_pages_per_route) {
  const int64_t cus = cu_count();
  const int64_t units = (int64_t)num_launch * num_kv_heads;
  const bool pairs_balance = max_pages_per_route <= kMinSplitPages || ((units + cus - 1) / cus) % 2 == 0;
  return !fp8 && !route_list && plan.max_chunks == 1 && max_pages_per_route <= kMaxPagesTwoUnit &&
                 units >= 2 * cus && pairs_balance
             ? 2
             : 1;
}

bool ordered_dispatch(const ChunkPlan& plan, int32_t num_launch, int32_t num_kv_heads,
                      int64_t slots) {
  const int64_t items = (int64_t)plan.max_chunks * num_kv_heads * num_launch;
  return plan.max_chunks > 1 && items >= 2 * slots && items <= kMaxOrderItems;
}

WorkspaceLayout workspace_layout(int32_t num_routes, int32_t num_kv_heads, int32_t group,
                                 int32_t max_chunks, bool ordered) {
  WorkspaceLayout l;
  const size_t units = (size_t)num_routes * num_kv_heads * max_chunks;
  const size_t recs = max_chunks > 1 ? units * group : 0;
  l.ml_off = 0;
  l.o_off = round_up(recs * 2 * sizeof(float), 256);
  l.order_off = l.o_off + round_up(recs * kDim * sizeof(float), 256);
  l.total = l.order_off + (ordered ? round_up((2 + 2 * units) * sizeof(uint32_t), 256) : 0);
  if (!ordered) l.order_off = 0;
  if (l.total < 256) l.total = 256;
  return l;
}

}  // namespace kf

extern "C" {

const char* kf_status_str(int status) {
  switch (status) {
    case KF_OK: return "ok";
    case KF_ERR_INVALID_ARG: return "invalid argument";
    case KF_ERR_UNSUPPORTED: return "unsupported shape or dtype";
    case KF_ERR_WORKSPACE: return "workspace missing or too small";
    case KF_ERR_HIP: return "HIP runtime error";
    case KF_ERR_CAPACITY: return "output array too small";
    case KF_ERR_INFEASIBLE: return "infeasible budget";
    case KF_ERR_HOST_MEMORY: return "host memory exhausted";
    case KF_ERR_SCRATCH_LIMIT: return "launch needs more than KF_SCRATCH_BYTES of scratch";
    default: return "unknown status";
  }
}

const char* kf_version(void) { return "kf 0.1 gfx950"; }

size_t kf_partial_attn_workspace_bytes(const kf_shape* shape, int32_t num_routes,
                                       int32_t max_pages_per_route) {
  if (check_shape(shape) != KF_OK || num_routes < 0 || max_pages_per_route < 0) return 0;
  if (num_routes > kf::kMaxLaunchRoutes || shape->num_kv_heads > kf::kMaxLaunchRoutes) return 0;
  const int32_t group = shape->num_q_heads / shape->num_kv_heads;
  const bool fp8 = shape->kv_dtype == KF_KV_FP8_E4M3;
  // The largest need of any launch of at most num_routes routes: fewer routes
  // may not fill the GPU and then split their units, so a workspace sized for
  // a whole route table must also serve a launch over a subset of it.  Both
  // readings of the page table (ragged routes or not) and both kinds of
  // launch (over the table, over a route list) are covered, so the size does
  // not depend on shape->num_page_ids, which grows with the table.
  // Launches whose units reach ranges_per_slot * slots keep every unit whole
  // and need no workspace, so at most that many route counts are visited.
  const int64_t slots = 2 * (int64_t)kf::cu_count();
  const int64_t split_units = kf::ranges_per_slot(fp8) * slots;
  size_t most = 256;
  for (int32_t m = 1; m <= num_routes && (int64_t)m * shape->num_kv_heads < split_units; ++m) {
    for (const bool ragged : {false, true})
      for (const bool listed : {false, true}) {
        const kf::ChunkPlan plan = kf::plan_for_slots(m, shape->num_kv_heads, max_pages_per_route,
                                                      ragged, fp8, slots, listed);
        const size_t t =
            kf::workspace_layout(m, shape->num_kv_heads, group, plan.max_chunks,
                                 kf::ordered_dispatch(plan, m, shape->num_kv_heads, slots))
                .total;
        if (t > most) most = t;
      }
  }
  return most;
}

int kf_partial_attn_plan(const kf_shape* shape, int32_t num_launch, int32_t max_pages_per_route,
                         int32_t route_list_launch, int32_t* chunk_pages, int32_t* max_chunks,
                         int32_t* units_per_wg) {
  const int st = check_shape(shape);
  if (st != KF_OK) return st;
  if (num_launch < 0 || max_pages_per_route < 0 || (route_list_launch != 0 && route_list_launch != 1))
    return KF_ERR_INVALID_ARG;
  if (num_launch > kf::kMaxLaunchRoutes || shape->num_kv_heads > kf::kMaxLaunchRoutes) return KF_ERR_UNSUPPORTED;
  const kf::ChunkPlan plan = kf::plan_chunks(
      num_launch, shape->num_kv_heads, max_pages_per_route,
      kf::ragged_table(shape->num_page_ids, num_launch, max_pages_per_route),
      shape->kv_dtype == KF_KV_FP8_E4M3, route_list_launch == 1);
  if (chunk_pages) *chunk_pages = plan.chunk_pages;
  if (max_chunks) *max_chunks = plan.max_chunks;
  if (units_per_wg)
    *units_per_wg = kf::units_per_workgroup(shape->kv_dtype == KF_KV_FP8_E4M3,
                                            route_list_launch == 1, plan, num_launch,
                                            shape->num_kv_heads, max_pages_per_route);
  return KF_OK;
}

}  // extern "C"

namespace {

// Host checks of kf_kv_append; fills the kernel arguments.
int prepare_append(const kf_shape* shape, void* k_pool, void* v_pool, float* k_scale,
                   float* v_scale, const void* k_new, const void* v_new, kf_route* routes,
                   int32_t num_routes, const int32_t* tail_route, const int32_t* page_ids,
                   int32_t* err_flags, kf::AppendArgs& a) {
  int st = check_shape(shape);
  if (st != KF_OK) return st;
  if (num_routes < 0) return KF_ERR_INVALID_ARG;
  if (shape->num_seqs == 0) return KF_OK;
  const bool fp8 = shape->kv_dtype == KF_KV_FP8_E4M3;
  if (!k_pool || !v_pool || !k_new || !v_new || !tail_route || !err_flags ||
      (num_routes > 0 && !routes) || (shape->num_page_ids > 0 && !page_ids))
    return KF_ERR_INVALID_ARG;
  if (fp8 && (!k_scale || !v_scale)) return KF_ERR_INVALID_ARG;
  const void* ptrs[] = {k_pool, v_pool, k_scale, v_scale, k_new, v_new,
                        routes, tail_route, page_ids, err_flags};
  for (const void* p : ptrs)
    if (p && !aligned(p, 4)) return KF_ERR_INVALID_ARG;
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.k_new = static_cast<const uint16_t*>(k_new);
  a.v_new = static_cast<const uint16_t*>(v_new);
  a.routes = routes;
  a.tail_route = tail_route;
  a.page_ids = page_ids;
  a.err_flags = err_flags;
  a.num_seqs = shape->num_seqs;
  a.num_kv_heads = shape->num_kv_heads;
  a.num_routes = num_routes;
  a.num_pages = shape->num_pages;
  a.num_page_ids = shape->num_page_ids;
  a.head_major = shape->kv_layout == KF_KV_HEAD_MAJOR;
  return KF_OK;
}

// Host checks of kf_partial_attn / kf_partial_attn_subset; fills the kernel
// arguments (a.num_units_routes == 0: nothing to launch).
int prepare_partial(const kf_shape* shape, const void* q, const void* k_pool, const void* v_pool,
                    const float* k_scale, const float* v_scale, const kf_route* routes,
                    int32_t num_routes, const int32_t* route_list, int32_t num_launch,
                    int32_t max_pages_per_route, const int32_t* page_ids, float* o_part,
                    float* lse_part, void* workspace, size_t workspace_bytes, int32_t* err_flags,
                    kf::PartialArgs& a) {
  int st = check_shape(shape);
  if (st != KF_OK) return st;
  if (num_routes < 0 || num_launch < 0 || max_pages_per_route < 0) return KF_ERR_INVALID_ARG;
  if (num_launch == 0) return KF_OK;
  if (num_launch > kf::kMaxLaunchRoutes || shape->num_kv_heads > kf::kMaxLaunchRoutes) return KF_ERR_UNSUPPORTED;
  const bool fp8 = shape->kv_dtype == KF_KV_FP8_E4M3;
  if (!q || !k_pool || !v_pool || !routes || !o_part || !lse_part || !err_flags ||
      (shape->num_page_ids > 0 && !page_ids))
    return KF_ERR_INVALID_ARG;
  if (fp8 && (!k_scale || !v_scale)) return KF_ERR_INVALID_ARG;
  if (!aligned(q, 16) || !aligned(k_pool, 16) || !aligned(v_pool, 16) || !aligned(o_part, 16))
    return KF_ERR_INVALID_ARG;
  const void* p4[] = {k_scale, v_scale, routes, route_list, page_ids, lse_part, err_flags};
  for (const void* p : p4)
    if (p && !aligned(p, 4)) return KF_ERR_INVALID_ARG;
  const int32_t group = shape->num_q_heads / shape->num_kv_heads;
  const kf::ChunkPlan plan = kf::plan_chunks(
      num_launch, shape->num_kv_heads, max_pages_per_route,
      kf::ragged_table(shape->num_page_ids, num_launch, max_pages_per_route),
      shape->kv_dtype == KF_KV_FP8_E4M3, route_list != nullptr);
  const bool ordered =
      kf::ordered_dispatch(plan, num_launch, shape->num_kv_heads, 2 * (int64_t)kf::cu_count());
  const kf::WorkspaceLayout l =
      kf::workspace_layout(num_launch, shape->num_kv_heads, group, plan.max_chunks, ordered);
  if (!workspace || !aligned(workspace, 256) || workspace_bytes < l.total) return KF_ERR_WORKSPACE;

  a.q = static_cast<const uint16_t*>(q);
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.k_scale = k_scale;
  a.v_scale = v_scale;
  a.routes = routes;
  a.route_list = route_list;
  a.page_ids = page_ids;
  a.o_part = o_part;
  a.lse_part = lse_part;
  char* ws = static_cast<char*>(workspace);
  a.ws_ml = reinterpret_cast<float*>(ws + l.ml_off);
  a.ws_o = reinterpret_cast<float*>(ws + l.o_off);
  a.order = ordered ? reinterpret_cast<uint32_t*>(ws + l.order_off) : nullptr;
  a.err_flags = err_flags;
  a.num_seqs = shape->num_seqs;
  a.num_q_heads = shape->num_q_heads;
  a.num_kv_heads = shape->num_kv_heads;
  a.group = group;
  a.num_routes = num_routes;
  a.max_pages_per_route = max_pages_per_route;
  a.num_units_routes = num_launch;
  a.chunk_pages = plan.chunk_pages;
  a.max_chunks = plan.max_chunks;
  a.units_per_wg = kf::units_per_workgroup(fp8, route_list != nullptr, plan, num_launch,
                                           shape->num_kv_heads, max_pages_per_route);
  a.num_pages = shape->num_pages;
  a.num_page_ids = shape->num_page_ids;
  a.head_major = shape->kv_layout == KF_KV_HEAD_MAJOR;
  a.scale_log2 = (float)((double)shape->scale * 1.4426950408889634074);
  return KF_OK;
}

int partial_attn_impl(const kf_shape* shape, const void* q, const void* k_pool, const void* v_pool,
                      const float* k_scale, const float* v_scale, const kf_route* routes,
                      int32_t num_routes, const int32_t* route_list, int32_t num_launch,
                      int32_t max_pages_per_route, const int32_t* page_ids, float* o_part,
                      float* lse_part, void* workspace, size_t workspace_bytes,
                      int32_t* err_flags, void* stream) {
  kf::PartialArgs a{};
  const int st = prepare_partial(shape, q, k_pool, v_pool, k_scale, v_scale, routes, num_routes,
                                 route_list, num_launch, max_pages_per_route, page_ids, o_part,
                                 lse_part, workspace, workspace_bytes, err_flags, a);
  if (st != KF_OK || a.num_units_routes == 0) return st;
  return kf::launch_partial(a, shape->kv_dtype == KF_KV_FP8_E4M3, as_stream(stream)) == hipSuccess
             ? KF_OK
             : KF_ERR_HIP;
}

// Host checks of kf_merge_partials; fills the kernel arguments.
int prepare_merge(int32_t num_seqs, int32_t num_routes, int32_t num_q_heads, int32_t head_dim,
                  const float* o_part, const float* lse_part, const int32_t* seq_route_begin,
                  float* out, float* lse_out, int32_t* err_flags, kf::MergeArgs& a) {
  if (num_seqs < 0 || num_routes < 0 || num_q_heads <= 0) return KF_ERR_INVALID_ARG;
  if (head_dim != KF_HEAD_DIM) return KF_ERR_UNSUPPORTED;
  if (num_seqs == 0) return KF_OK;
  if (num_seqs > 65535 || num_q_heads > 65535) return KF_ERR_UNSUPPORTED;
  if (!seq_route_begin || !out || !lse_out || !err_flags ||
      (num_routes > 0 && (!o_part || !lse_part)))
    return KF_ERR_INVALID_ARG;
  if ((o_part && !aligned(o_part, 8)) || !aligned(out, 8)) return KF_ERR_INVALID_ARG;
  const void* p4[] = {lse_part, seq_route_begin, lse_out, err_flags};
  for (const void* p : p4)
    if (p && !aligned(p, 4)) return KF_ERR_INVALID_ARG;
  a.o_part = o_part;
  a.lse_part = lse_part;
  a.seq_route_begin = seq_route_begin;
  a.out = out;
  a.lse_out = lse_out;
  a.err_flags = err_flags;
  a.num_seqs = num_seqs;
  a.num_routes = num_routes;
  a.num_q_heads = num_q_heads;
  return KF_OK;
}

// The decode step of kf_decode_step (workspace given) and
// kf_decode_step_no_alloc (use_scratch: the device's scratch array instead).
int decode_step_impl(const kf_shape* shape, const void* q, void* k_pool, void* v_pool,
                     float* k_scale, float* v_scale, const void* k_new, const void* v_new,
                     kf_route* routes, int32_t num_routes, const int32_t* tail_route,
                     int32_t max_pages_per_route, const int32_t* page_ids,
                     const int32_t* seq_route_begin, float* o_part, float* lse_part, float* out,
                     float* lse_out, void* workspace, size_t workspace_bytes, bool use_scratch,
                     int32_t* err_flags, void* stream) {
  kf::AppendArgs ap{};
  kf::PartialArgs pa{};
  kf::MergeArgs ma{};
  int st = prepare_append(shape, k_pool, v_pool, k_scale, v_scale, k_new, v_new, routes,
                          num_routes, tail_route, page_ids, err_flags, ap);
  if (st != KF_OK) return st;
  // The scratch array's size is checked like a workspace's, against a
  // stand-in base address; the array's own address is taken only once every
  // host check has passed.
  char* const kStandIn = reinterpret_cast<char*>((uintptr_t)256);
  if (use_scratch) {
    workspace = kStandIn;
    workspace_bytes = KF_SCRATCH_BYTES;
  }
  st = prepare_partial(shape, q, k_pool, v_pool, k_scale, v_scale, routes, num_routes, nullptr,
                       num_routes, max_pages_per_route, page_ids, o_part, lse_part, workspace,
                       workspace_bytes, err_flags, pa);
  // the workspace is the last check of prepare_partial: a scratch array too
  // small for this launch is reported after every argument check has passed
  const bool over_scratch = use_scratch && st == KF_ERR_WORKSPACE;
  if (st != KF_OK && !over_scratch) return st;
  st = prepare_merge(shape->num_seqs, num_routes, shape->num_q_heads, shape->head_dim, o_part,
                     lse_part, seq_route_begin, out, lse_out, err_flags, ma);
  if (st != KF_OK) return st;
  if (over_scratch) return KF_ERR_SCRATCH_LIMIT;
  if (shape->num_seqs == 0) return KF_OK;
  if (use_scratch && num_routes > 0) {
    void* base = nullptr;
    if (kf::scratch_address(&base) != hipSuccess) return KF_ERR_HIP;
    const uintptr_t b = reinterpret_cast<uintptr_t>(base), s0 = reinterpret_cast<uintptr_t>(kStandIn);
    pa.ws_ml = reinterpret_cast<float*>(b + (reinterpret_cast<uintptr_t>(pa.ws_ml) - s0));
    pa.ws_o = reinterpret_cast<float*>(b + (reinterpret_cast<uintptr_t>(pa.ws_o) - s0));
    if (pa.order)
      pa.order = reinterpret_cast<uint32_t*>(b + (reinterpret_cast<uintptr_t>(pa.order) - s0));
  }
  const hipStream_t s = as_stream(stream);
  const bool fp8 = shape->kv_dtype == KF_KV_FP8_E4M3;
  if (num_routes == 0) {  // nothing to attend: the append kernel raises the flags
    if (kf::launch_append(ap, fp8, s) != hipSuccess) return KF_ERR_HIP;
    return kf::launch_merge(ma, s) == hipSuccess ? KF_OK : KF_ERR_HIP;
  }
  pa.k_new = ap.k_new;
  pa.v_new = ap.v_new;
  pa.tail_route = tail_route;
  pa.k_pool_w = k_pool;
  pa.v_pool_w = v_pool;
  pa.k_scale_w = k_scale;
  pa.v_scale_w = v_scale;
  ma.routes = routes;
  ma.tail_route = tail_route;
  ma.page_ids = page_ids;
  ma.num_pages = shape->num_pages;
  ma.num_page_ids = shape->num_page_ids;
  if (kf::launch_partial(pa, fp8, s) != hipSuccess) return KF_ERR_HIP;
  return kf::launch_merge(ma, s) == hipSuccess ? KF_OK : KF_ERR_HIP;
}

}  // namespace

extern "C" {

int kf_kv_append(const kf_shape* shape, void* k_pool, void* v_pool, float* k_scale,
                 float* v_scale, const void* k_new, const void* v_new, kf_route* routes,
                 int32_t num_routes, const int32_t* tail_route, const int32_t* page_ids,
                 int32_t* err_flags, void* stream) {
  kf::AppendArgs a{};
  const int st = prepare_append(shape, k_pool, v_pool, k_scale, v_scale, k_new, v_new, routes,
                                num_routes, tail_route, page_ids, err_flags, a);
  if (st != KF_OK || shape->num_seqs == 0) return st;
  return kf::launch_append(a, shape->kv_dtype == KF_KV_FP8_E4M3, as_stream(stream)) == hipSuccess
             ? KF_OK
             : KF_ERR_HIP;
}

int kf_partial_attn(const kf_shape* shape, const void* q, const void* k_pool, const void* v_pool,
                    const float* k_scale, const float* v_scale, const kf_route* routes,
                    int32_t num_routes, int32_t max_pages_per_route, const int32_t* page_ids,
                    float* o_part, float* lse_part, void* workspace, size_t workspace_bytes,
                    int32_t* err_flags, void* stream) {
  return partial_attn_impl(shape, q, k_pool, v_pool, k_scale, v_scale, routes, num_routes,
                           nullptr, num_routes, max_pages_per_route, page_ids, o_part, lse_part,
                           workspace, workspace_bytes, err_flags, stream);
}

int kf_partial_attn_subset(const kf_shape* shape, const void* q, const void* k_pool,
                           const void* v_pool, const float* k_scale, const float* v_scale,
                           const kf_route* routes, int32_t num_routes, const int32_t* route_list,
                           int32_t num_list, int32_t max_pages_per_route, const int32_t* page_ids,
                           float* o_part, float* lse_part, void* workspace,
                           size_t workspace_bytes, int32_t* err_flags, void* stream) {
  if (num_list > 0 && !route_list) return KF_ERR_INVALID_ARG;
  return partial_attn_impl(shape, q, k_pool, v_pool, k_scale, v_scale, routes, num_routes,
                           route_list, num_list, max_pages_per_route, page_ids, o_part, lse_part,
                           workspace, workspace_bytes, err_flags, stream);
}

int kf_merge_partials(int32_t num_seqs, int32_t num_routes, int32_t num_q_heads, int32_t head_dim,
                      const float* o_part, const float* lse_part, const int32_t* seq_route_begin,
                      float* out, float* lse_out, int32_t* err_flags, void* stream) {
  kf::MergeArgs a{};
  const int st = prepare_merge(num_seqs, num_routes, num_q_heads, head_dim, o_part, lse_part,
                               seq_route_begin, out, lse_out, err_flags, a);
  if (st != KF_OK || num_seqs == 0) return st;
  return kf::launch_merge(a, as_stream(stream)) == hipSuccess ? KF_OK : KF_ERR_HIP;
}

int kf_debug_gather(const kf_shape* shape, const void* k_pool, const void* v_pool,
                    const kf_route* routes, int32_t num_routes, int32_t route,
                    int32_t max_pages_per_route, const int32_t* page_ids, int32_t max_tokens,
                    void* out_k, void* out_v, int32_t* err_flags, void* stream) {
  const int st = check_shape(shape);
  if (st != KF_OK) return st;
  if (num_routes < 0 || route < 0 || route >= num_routes || max_pages_per_route < 0 ||
      max_tokens < 0)
    return KF_ERR_INVALID_ARG;
  if (!k_pool || !v_pool || !routes || !err_flags || (shape->num_page_ids > 0 && !page_ids) ||
      (max_tokens > 0 && (!out_k || !out_v)))
    return KF_ERR_INVALID_ARG;
  const void* p4[] = {k_pool, v_pool, routes, page_ids, out_k, out_v, err_flags};
  for (const void* p : p4)
    if (p && !aligned(p, 4)) return KF_ERR_INVALID_ARG;
  if (max_tokens == 0) return KF_OK;
  kf::PartialArgs a{};
  a.k_pool = k_pool;
  a.v_pool = v_pool;
  a.routes = routes;
  a.page_ids = page_ids;
  a.err_flags = err_flags;
  a.num_seqs = shape->num_seqs;
  a.num_q_heads = shape->num_q_heads;
  a.num_kv_heads = shape->num_kv_heads;
  a.num_routes = num_routes;
  a.max_pages_per_route = max_pages_per_route;
  a.num_pages = shape->num_pages;
  a.num_page_ids = shape->num_page_ids;
  a.head_major = shape->kv_layout == KF_KV_HEAD_MAJOR;
  return kf::launch_gather(a, shape->kv_dtype == KF_KV_FP8_E4M3, route, max_tokens, out_k, out_v,
                           as_stream(stream)) == hipSuccess
             ? KF_OK
             : KF_ERR_HIP;
}

int kf_decode_step(const kf_shape* shape, const void* q, void* k_pool, void* v_pool,
                   float* k_scale, float* v_scale, const void* k_new, const void* v_new,
                   kf_route* routes, int32_t num_routes, const int32_t* tail_route,
                   int32_t max_pages_per_route, const int32_t* page_ids,
                   const int32_t* seq_route_begin, float* o_part, float* lse_part, float* out,
                   float* lse_out, void* workspace, size_t workspace_bytes, int32_t* err_flags,
                   void* stream) {
  return decode_step_impl(shape, q, k_pool, v_pool, k_scale, v_scale, k_new, v_new, routes,
                          num_routes, tail_route, max_pages_per_route, page_ids, seq_route_begin,
                          o_part, lse_part, out, lse_out, workspace, workspace_bytes, false,
                          err_flags, stream);
}

int kf_decode_step_no_alloc(const kf_shape* shape, const void* q, void* k_pool, void* v_pool,
                            float* k_scale, float* v_scale, const void* k_new,
                            const void* v_new, kf_route* routes, int32_t num_routes,
                            const int32_t* tail_route, int32_t max_pages_per_route,
                            const int32_t* page_ids, const int32_t* seq_route_begin,
                            float* o_part, float* lse_part, float* out, float* lse_out,
                            int32_t* err_flags, void* stream) {
  return decode_step_impl(shape, q, k_pool, v_pool, k_scale, v_scale, k_new, v_new, routes,
                          num_routes, tail_route, max_pages_per_route, page_ids, seq_route_begin,
                          o_part, lse_part, out, lse_out, nullptr, 0, true, err_flags, stream);
}

}  // extern "C"
