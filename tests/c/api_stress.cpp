// Host-only stress of the C-ABI layer (paper_2606_29207_amd/csrc/kf_api.cpp),
// built with g++ under AddressSanitizer and UndefinedBehaviorSanitizer
// against the HIP test double in tests/c/hipstub.  The kernel launchers are
// replaced by checkers: every launch the layer makes must fit the grid
// limits, cover the longest route with its page ranges, and stay inside the
// workspace it was given (the checker writes the first and last element of
// every workspace region, so an under-sized layout is an ASan error).
//
//   valid calls    random valid arguments: KF_OK, launches consistent
//   one mutation   a valid call with one argument broken: the documented
//                  status, and nothing launched
//   fuzz           arbitrary arguments: a known status, no sanitizer report
//   plan/workspace kf_partial_attn_plan and the workspace query over random
//                  and extreme sizes and device CU counts; a workspace of the
//                  queried size is always accepted, and the query stays fast
//
// Usage: api_stress [iterations]; prints "api_stress ok" on success.
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include <chrono>
#include <random>
#include <vector>

#include "kf.h"
#include "kf_internal.h"

// ------------------------------------------------------------- HIP double
static int g_device = 0;
static bool g_no_device = false;
static const int kCus[8] = {256, 304, 80, 1, 1024, 32, 120, 228};

hipError_t hipGetDevice(int* device) {
  if (g_no_device) return hipErrorNoDevice;
  *device = g_device;
  return hipSuccess;
}
hipError_t hipGetLastError(void) { return hipSuccess; }
hipError_t hipDeviceGetAttribute(int* value, hipDeviceAttribute_t attr, int device) {
  if (attr != hipDeviceAttributeMultiprocessorCount || device < 0 || device >= 8)
    return hipErrorInvalidValue;
  *value = kCus[device];
  return hipSuccess;
}

// Whether a launch with this plan runs in a computed dispatch order on the
// current fake device (two resident workgroups per CU).
static int64_t fake_slots() { return 2 * (int64_t)(g_no_device ? 256 : kCus[g_device]); }
static bool ordered(int32_t cp, int32_t mc, int32_t routes, int32_t heads) {
  return kf::ordered_dispatch(kf::ChunkPlan{cp, mc}, routes, heads, fake_slots());
}

// ------------------------------------------------------- launch checkers
static int g_launches = 0;
static bool g_fail_launch = false;
static unsigned char* g_ws = nullptr;  // the real host workspace of the current call, if any
static size_t g_ws_bytes = 0;
static long g_errors = 0;

#define CHECK(cond, ...)                                  \
  do {                                                    \
    if (!(cond)) {                                        \
      ++g_errors;                                         \
      if (g_errors < 20) {                                \
        fprintf(stderr, "%s:%d: %s: ", __FILE__, __LINE__, #cond); \
        fprintf(stderr, __VA_ARGS__);                     \
        fprintf(stderr, "\n");                            \
      }                                                   \
    }                                                     \
  } while (0)

static void touch(void* p) {
  // a write the sanitizer checks when p lies in the real workspace buffer
  unsigned char* c = static_cast<unsigned char*>(p);
  if (g_ws && c >= g_ws && c < g_ws + g_ws_bytes + 4096) *c = 0x5a;
  else if (g_ws) CHECK(false, "workspace pointer %p outside [%p, +%zu)", p, (void*)g_ws, g_ws_bytes);
}

namespace kf {

hipError_t launch_append(const AppendArgs& a, bool fp8, hipStream_t) {
  ++g_launches;
  CHECK(a.num_seqs >= 1 && a.num_seqs <= 2147483647, "append grid %d", a.num_seqs);
  CHECK(a.k_pool && a.v_pool && a.k_new && a.v_new && a.tail_route && a.err_flags, "append ptrs");
  CHECK(!fp8 || (a.k_scale && a.v_scale), "fp8 append without scales");
  CHECK(a.num_routes == 0 || a.routes, "append routes");
  return g_fail_launch ? hipErrorInvalidValue : hipSuccess;
}

hipError_t launch_partial(const PartialArgs& a, bool fp8, hipStream_t) {
  ++g_launches;
  CHECK(a.num_units_routes >= 1 && a.num_units_routes <= 65535, "grid z %d", a.num_units_routes);
  CHECK(a.num_kv_heads >= 1 && a.num_kv_heads <= 65535, "grid y %d", a.num_kv_heads);
  CHECK(a.group >= 1 && a.group <= KF_MAX_GROUP && a.group * a.num_kv_heads == a.num_q_heads,
        "group %d", a.group);
  CHECK(a.max_chunks >= 1 && a.max_chunks <= 65535, "grid x %d", a.max_chunks);
  CHECK(a.chunk_pages >= 1, "chunk_pages %d", a.chunk_pages);
  if (a.chunk_pages >= 1) {
    const long long need = ((long long)a.max_pages_per_route + a.chunk_pages - 1) / a.chunk_pages;
    CHECK(need <= a.max_chunks, "ranges do not cover %d pages: %d x %d", a.max_pages_per_route,
          a.max_chunks, a.chunk_pages);
  }
  CHECK(a.units_per_wg == 1 || a.units_per_wg == 2, "units_per_wg %d", a.units_per_wg);
  if (a.units_per_wg == 2)
    CHECK(!fp8 && a.max_chunks == 1 && !a.route_list, "two-unit mode on a split or listed launch");
  CHECK(a.q && a.k_pool && a.v_pool && a.routes && a.o_part && a.lse_part && a.err_flags,
        "partial ptrs");
  CHECK(!fp8 || (a.k_scale && a.v_scale), "fp8 partial without scales");
  CHECK(isfinite(a.scale_log2), "scale_log2");
  if (a.k_new) CHECK(a.v_new && a.tail_route && a.k_pool_w && a.v_pool_w, "fused ptrs");
  if (a.max_chunks > 1) {
    const size_t recs = (size_t)a.num_units_routes * a.num_kv_heads * a.max_chunks * a.group;
    touch(a.ws_ml);
    touch(a.ws_ml + recs * 2 - 1);
    touch(a.ws_o);
    touch(a.ws_o + recs * kDim - 1);
    if (g_ws)
      CHECK((unsigned char*)(a.ws_o + recs * kDim) <= g_ws + g_ws_bytes,
            "workspace needs %zu records, has %zu bytes", recs, g_ws_bytes);
  }
  const size_t items = (size_t)a.num_units_routes * a.num_kv_heads * a.max_chunks;
  CHECK(!a.order == !kf::ordered_dispatch(kf::ChunkPlan{a.chunk_pages, a.max_chunks},
                                          a.num_units_routes, a.num_kv_heads, fake_slots()),
        "dispatch order %p for %zu items", (const void*)a.order, items);
  if (a.order) {
    CHECK(a.max_chunks > 1 && a.units_per_wg == 1, "dispatch order of an unsplit launch");
    const size_t recs = items * a.group;
    touch(a.order);
    touch(a.order + 2 + 2 * items - 1);
    CHECK((const unsigned char*)a.order >= (const unsigned char*)(a.ws_o + recs * kDim),
          "dispatch order over the records");
    if (g_ws)
      CHECK((unsigned char*)(a.order + 2 + 2 * items) <= g_ws + g_ws_bytes,
            "dispatch order of %zu items past the workspace of %zu bytes", items, g_ws_bytes);
  }
  return g_fail_launch ? hipErrorInvalidValue : hipSuccess;
}

hipError_t launch_merge(const MergeArgs& a, hipStream_t) {
  ++g_launches;
  CHECK(a.num_seqs >= 1 && a.num_seqs <= 65535 && a.num_q_heads >= 1 && a.num_q_heads <= 65535,
        "merge grid %d x %d", a.num_q_heads, a.num_seqs);
  CHECK(a.seq_route_begin && a.out && a.lse_out && a.err_flags, "merge ptrs");
  CHECK(a.num_routes == 0 || (a.o_part && a.lse_part), "merge partials");
  if (a.tail_route) CHECK(a.routes, "fused merge without routes");
  return g_fail_launch ? hipErrorInvalidValue : hipSuccess;
}

// The scratch array of kf_decode_step_no_alloc: a host buffer of its size,
// made the checked workspace of the call that asks for it.
static std::vector<unsigned char> scratch_buf;
hipError_t scratch_address(void** out) {
  if (scratch_buf.empty()) scratch_buf.resize(KF_SCRATCH_BYTES + 256);
  uintptr_t base = ((uintptr_t)scratch_buf.data() + 255) & ~(uintptr_t)255;
  g_ws = reinterpret_cast<unsigned char*>(base);
  g_ws_bytes = KF_SCRATCH_BYTES;
  *out = g_ws;
  return hipSuccess;
}

hipError_t launch_gather(const PartialArgs& a, bool, int route, int max_tokens, void* out_k,
                         void* out_v, hipStream_t) {
  ++g_launches;
  CHECK(max_tokens >= 1 && route >= 0 && route < a.num_routes, "gather %d %d", max_tokens, route);
  CHECK(out_k && out_v && a.k_pool && a.v_pool && a.routes && a.err_flags, "gather ptrs");
  return g_fail_launch ? hipErrorInvalidValue : hipSuccess;
}

}  // namespace kf

// ------------------------------------------------------------- arguments
static std::mt19937_64 rng(12345);
static int64_t rnd(int64_t lo, int64_t hi) {  // inclusive
  return std::uniform_int_distribution<int64_t>(lo, hi)(rng);
}
static bool coin(double p) { return std::uniform_real_distribution<double>(0, 1)(rng) < p; }

// Non-null stand-ins, 256-byte aligned, never dereferenced by the layer.
static void* fake(int k) { return reinterpret_cast<void*>((uintptr_t)(0x100000 + 0x1000 * k)); }
static void* misalign(void* p, int by) { return reinterpret_cast<void*>((uintptr_t)p + by); }

struct Call {
  kf_shape s;
  void *q, *k, *v, *ks, *vs, *kn, *vn, *routes, *tail, *pids, *srb, *o, *lse, *out, *lse_out,
      *flags, *list;
  int32_t R, maxp, nlist;
  void* ws;
  size_t wsb;
};

static kf_shape valid_shape() {
  kf_shape s;
  const int32_t H = (int32_t)(coin(0.05) ? rnd(1, 70) : (int)(1 << rnd(0, 4)));
  const int32_t G = (int32_t)rnd(1, KF_MAX_GROUP);
  s.num_seqs = (int32_t)(coin(0.05) ? rnd(1, 65535) : rnd(1, 128));
  s.num_q_heads = H * G;
  s.num_kv_heads = H;
  s.head_dim = KF_HEAD_DIM;
  s.page_size = KF_PAGE_SIZE;
  s.kv_dtype = coin(0.5) ? KF_KV_BF16 : KF_KV_FP8_E4M3;
  s.num_pages = (int32_t)rnd(1, 1 << 24);
  s.num_page_ids = (int32_t)(coin(0.1) ? 0 : rnd(0, 1 << 26));
  s.scale = 0.0883883f;
  s.kv_layout = coin(0.5) ? KF_KV_PAGE_MAJOR : KF_KV_HEAD_MAJOR;
  return s;
}

static Call valid_call() {
  Call c;
  memset(&c, 0, sizeof c);
  c.s = valid_shape();
  void** ptrs[] = {&c.q, &c.k, &c.v, &c.kn, &c.vn, &c.routes, &c.tail, &c.pids, &c.srb,
                   &c.o, &c.lse, &c.out, &c.lse_out, &c.flags, &c.list};
  int k = 0;
  for (void** p : ptrs) *p = fake(++k);
  if (c.s.kv_dtype == KF_KV_FP8_E4M3) {
    c.ks = fake(++k);
    c.vs = fake(++k);
  }
  c.R = (int32_t)(coin(0.1) ? rnd(1, 65535) : rnd(1, 600));
  c.maxp = (int32_t)(coin(0.1) ? rnd(0, 2147483647) : rnd(0, 9000));
  c.nlist = (int32_t)rnd(1, c.R);
  if (c.s.num_page_ids == 0) c.pids = coin(0.5) ? nullptr : c.pids;
  return c;
}

// Workspace of the queried size as a real host buffer when it is small
// enough, else a stand-in; returns the queried size.
static std::vector<unsigned char> ws_buf;
static size_t attach_workspace(Call& c, int32_t routes_for_query) {
  const size_t n = kf_partial_attn_workspace_bytes(&c.s, routes_for_query, c.maxp);
  CHECK(n >= 256 && n % 256 == 0, "workspace query %zu for R=%d maxp=%d H=%d", n,
        routes_for_query, c.maxp, c.s.num_kv_heads);
  if (n <= (64u << 20)) {
    ws_buf.assign(n + 256, 0);
    uintptr_t base = ((uintptr_t)ws_buf.data() + 255) & ~(uintptr_t)255;
    g_ws = reinterpret_cast<unsigned char*>(base);
    g_ws_bytes = n;
    c.ws = g_ws;
  } else {
    g_ws = nullptr;
    g_ws_bytes = 0;
    c.ws = fake(200);
  }
  c.wsb = n;
  return n;
}

static int call_partial(const Call& c) {
  return kf_partial_attn(&c.s, c.q, c.k, c.v, (const float*)c.ks, (const float*)c.vs,
                         (const kf_route*)c.routes, c.R, c.maxp, (const int32_t*)c.pids,
                         (float*)c.o, (float*)c.lse, c.ws, c.wsb, (int32_t*)c.flags, nullptr);
}
static int call_subset(const Call& c) {
  return kf_partial_attn_subset(&c.s, c.q, c.k, c.v, (const float*)c.ks, (const float*)c.vs,
                                (const kf_route*)c.routes, c.R, (const int32_t*)c.list, c.nlist,
                                c.maxp, (const int32_t*)c.pids, (float*)c.o, (float*)c.lse, c.ws,
                                c.wsb, (int32_t*)c.flags, nullptr);
}
static int call_step(const Call& c) {
  return kf_decode_step(&c.s, c.q, c.k, c.v, (float*)c.ks, (float*)c.vs, c.kn, c.vn,
                        (kf_route*)c.routes, c.R, (const int32_t*)c.tail, c.maxp,
                        (const int32_t*)c.pids, (const int32_t*)c.srb, (float*)c.o, (float*)c.lse,
                        (float*)c.out, (float*)c.lse_out, c.ws, c.wsb, (int32_t*)c.flags, nullptr);
}
static int call_step_no_alloc(const Call& c) {
  return kf_decode_step_no_alloc(&c.s, c.q, c.k, c.v, (float*)c.ks, (float*)c.vs, c.kn, c.vn,
                                 (kf_route*)c.routes, c.R, (const int32_t*)c.tail, c.maxp,
                                 (const int32_t*)c.pids, (const int32_t*)c.srb, (float*)c.o,
                                 (float*)c.lse, (float*)c.out, (float*)c.lse_out,
                                 (int32_t*)c.flags, nullptr);
}
static int call_append(const Call& c) {
  return kf_kv_append(&c.s, c.k, c.v, (float*)c.ks, (float*)c.vs, c.kn, c.vn, (kf_route*)c.routes,
                      c.R, (const int32_t*)c.tail, (const int32_t*)c.pids, (int32_t*)c.flags,
                      nullptr);
}
static int call_merge(const Call& c) {
  return kf_merge_partials(c.s.num_seqs, c.R, c.s.num_q_heads, c.s.head_dim, (const float*)c.o,
                           (const float*)c.lse, (const int32_t*)c.srb, (float*)c.out,
                           (float*)c.lse_out, (int32_t*)c.flags, nullptr);
}
static int call_gather(const Call& c) {
  const int32_t route = c.nlist > -2147483647 ? c.nlist - 1 : 0;
  return kf_debug_gather(&c.s, c.k, c.v, (const kf_route*)c.routes, c.R, route, c.maxp,
                         (const int32_t*)c.pids, (int32_t)(c.maxp % 4096) + 1, c.o, c.out,
                         (int32_t*)c.flags, nullptr);
}

static bool known_status(int st) { return st <= 0 && st >= KF_ERR_SCRATCH_LIMIT; }

// ---------------------------------------------------------------- checks
typedef int (*Entry)(const Call&);
struct EntryInfo {
  const char* name;
  Entry fn;
  int launches;  // of a valid call with work
  bool uses_ws;
};
static const EntryInfo kEntries[] = {
    {"kf_partial_attn", call_partial, -1, true}, {"kf_partial_attn_subset", call_subset, -1, true},
    {"kf_decode_step", call_step, 2, true},      {"kf_kv_append", call_append, 1, false},
    {"kf_merge_partials", call_merge, 1, false}, {"kf_debug_gather", call_gather, 1, false},
};
// with the no-alloc step, whose valid calls may be refused for size (above)
static const EntryInfo kMutEntries[] = {
    {"kf_partial_attn", call_partial, -1, true}, {"kf_partial_attn_subset", call_subset, -1, true},
    {"kf_decode_step", call_step, 2, true},      {"kf_kv_append", call_append, 1, false},
    {"kf_merge_partials", call_merge, 1, false}, {"kf_debug_gather", call_gather, 1, false},
    {"kf_decode_step_no_alloc", call_step_no_alloc, 2, false},
};

static void valid_calls(int iters) {
  for (int it = 0; it < iters; ++it) {
    g_device = (int)rnd(0, 7);
    for (const EntryInfo& e : kEntries) {
      Call c = valid_call();
      if (e.fn == call_merge) c.s.num_q_heads = (int32_t)rnd(1, 4096);
      if (e.uses_ws) attach_workspace(c, e.fn == call_subset ? (coin(0.5) ? c.nlist : c.R) : c.R);
      g_launches = 0;
      const int st = e.fn(c);
      CHECK(st == KF_OK, "%s valid call -> %d (R=%d maxp=%d H=%d G=%d)", e.name, st, c.R, c.maxp,
            c.s.num_kv_heads, c.s.num_q_heads / c.s.num_kv_heads);
      if (e.launches > 0) CHECK(g_launches == e.launches, "%s made %d launches", e.name, g_launches);
      if (e.launches < 0) CHECK(g_launches == 1 || g_launches == 0, "%s launches %d", e.name, g_launches);
      g_fail_launch = true;
      g_launches = 0;
      const int st2 = e.fn(c);
      g_fail_launch = false;
      CHECK(st2 == KF_ERR_HIP, "%s with a refused launch -> %d", e.name, st2);
      g_ws = nullptr;
    }
  }
}

// kf_decode_step_no_alloc on valid arguments: KF_OK and two launches when the
// launch's workspace need fits the scratch array, else KF_ERR_SCRATCH_LIMIT
// before anything is launched.
static void valid_no_alloc(int iters) {
  long fits = 0, refused = 0;
  for (int it = 0; it < iters; ++it) {
    g_device = (int)rnd(0, 7);
    Call c = valid_call();
    int32_t cp = 0, mc = 0, up = 0;
    CHECK(kf_partial_attn_plan(&c.s, c.R, c.maxp, 0, &cp, &mc, &up) == KF_OK, "plan");
    const size_t need =
        kf::workspace_layout(c.R, c.s.num_kv_heads, c.s.num_q_heads / c.s.num_kv_heads, mc,
                             ordered(cp, mc, c.R, c.s.num_kv_heads))
            .total;
    g_launches = 0;
    g_ws = nullptr;
    const int st = call_step_no_alloc(c);
    if (need <= KF_SCRATCH_BYTES) {
      CHECK(st == KF_OK && g_launches == 2, "no-alloc step -> %d, %d launches (need %zu)", st,
            g_launches, need);
      ++fits;
    } else {
      CHECK(st == KF_ERR_SCRATCH_LIMIT && g_launches == 0, "no-alloc step over the limit -> %d",
            st);
      ++refused;
    }
    g_fail_launch = true;
    const int st2 = call_step_no_alloc(c);
    g_fail_launch = false;
    CHECK(st2 == (need <= KF_SCRATCH_BYTES ? KF_ERR_HIP : KF_ERR_SCRATCH_LIMIT),
          "refused launch -> %d", st2);
    g_ws = nullptr;
  }
  CHECK(fits > 0 && refused > 0, "no-alloc sweep saw %ld fitting and %ld refused launches", fits,
        refused);
}

// One broken argument at a time: the status the header documents, no launch.
static void one_mutation(int iters) {
  struct Mut {
    const char* what;
    int expect;
    void (*apply)(Call&);
  };
  static const Mut muts[] = {
      {"null shape", KF_ERR_INVALID_ARG, nullptr},
      {"num_q_heads % num_kv_heads", KF_ERR_INVALID_ARG,
       [](Call& c) { c.s.num_kv_heads = 3; c.s.num_q_heads = 4; }},
      {"negative num_seqs", KF_ERR_INVALID_ARG, [](Call& c) { c.s.num_seqs = -1; }},
      {"zero kv heads", KF_ERR_INVALID_ARG, [](Call& c) { c.s.num_kv_heads = 0; }},
      {"no pages", KF_ERR_INVALID_ARG, [](Call& c) { c.s.num_pages = 0; }},
      {"negative page ids", KF_ERR_INVALID_ARG, [](Call& c) { c.s.num_page_ids = -5; }},
      {"group > 16", KF_ERR_UNSUPPORTED,
       [](Call& c) { c.s.num_kv_heads = 1; c.s.num_q_heads = 17; }},
      {"head_dim 64", KF_ERR_UNSUPPORTED, [](Call& c) { c.s.head_dim = 64; }},
      {"page size 32", KF_ERR_UNSUPPORTED, [](Call& c) { c.s.page_size = 32; }},
      {"dtype 7", KF_ERR_UNSUPPORTED, [](Call& c) { c.s.kv_dtype = 7; }},
      {"layout 2", KF_ERR_UNSUPPORTED, [](Call& c) { c.s.kv_layout = 2; }},
      {"NaN scale", KF_ERR_INVALID_ARG, [](Call& c) { c.s.scale = NAN; }},
      {"infinite scale", KF_ERR_INVALID_ARG, [](Call& c) { c.s.scale = INFINITY; }},
      {"null k_pool", KF_ERR_INVALID_ARG, [](Call& c) { c.k = nullptr; }},
      {"null v_pool", KF_ERR_INVALID_ARG, [](Call& c) { c.v = nullptr; }},
      {"null err_flags", KF_ERR_INVALID_ARG, [](Call& c) { c.flags = nullptr; }},
      {"null page_ids", KF_ERR_INVALID_ARG,
       [](Call& c) { c.s.num_page_ids = 10; c.pids = nullptr; }},
      {"misaligned err_flags", KF_ERR_INVALID_ARG, [](Call& c) { c.flags = misalign(c.flags, 2); }},
      {"misaligned page_ids", KF_ERR_INVALID_ARG,
       [](Call& c) { c.s.num_page_ids = 10; c.pids = misalign(c.pids, 1); }},
      {"fp8 without k_scale", KF_ERR_INVALID_ARG,
       [](Call& c) { c.s.kv_dtype = KF_KV_FP8_E4M3; c.ks = nullptr; c.vs = fake(90); }},
      {"fp8 without v_scale", KF_ERR_INVALID_ARG,
       [](Call& c) { c.s.kv_dtype = KF_KV_FP8_E4M3; c.vs = nullptr; c.ks = fake(91); }},
  };
  // Checks that only some entry points make.
  static const Mut attn_muts[] = {
      {"null q", KF_ERR_INVALID_ARG, [](Call& c) { c.q = nullptr; }},
      {"null o_part", KF_ERR_INVALID_ARG, [](Call& c) { c.o = nullptr; }},
      {"null lse_part", KF_ERR_INVALID_ARG, [](Call& c) { c.lse = nullptr; }},
      {"null routes", KF_ERR_INVALID_ARG, [](Call& c) { c.routes = nullptr; }},
      {"q misaligned to 16", KF_ERR_INVALID_ARG, [](Call& c) { c.q = misalign(c.q, 8); }},
      {"k_pool misaligned to 16", KF_ERR_INVALID_ARG, [](Call& c) { c.k = misalign(c.k, 4); }},
      {"o_part misaligned to 16", KF_ERR_INVALID_ARG, [](Call& c) { c.o = misalign(c.o, 4); }},
      {"lse_part misaligned", KF_ERR_INVALID_ARG, [](Call& c) { c.lse = misalign(c.lse, 2); }},
      {"negative max pages", KF_ERR_INVALID_ARG, [](Call& c) { c.maxp = -1; }},
      {"65536 routes", KF_ERR_UNSUPPORTED, [](Call& c) { c.R = 65536; c.nlist = 65536; }},
      {"null workspace", KF_ERR_WORKSPACE, [](Call& c) { c.ws = nullptr; }},
      {"workspace misaligned", KF_ERR_WORKSPACE, [](Call& c) { c.ws = misalign(c.ws, 128); }},
  };
  static const Mut step_muts[] = {
      {"null k_new", KF_ERR_INVALID_ARG, [](Call& c) { c.kn = nullptr; }},
      {"null v_new", KF_ERR_INVALID_ARG, [](Call& c) { c.vn = nullptr; }},
      {"null tail_route", KF_ERR_INVALID_ARG, [](Call& c) { c.tail = nullptr; }},
      {"misaligned k_new", KF_ERR_INVALID_ARG, [](Call& c) { c.kn = misalign(c.kn, 2); }},
      {"null seq_route_begin", KF_ERR_INVALID_ARG, [](Call& c) { c.srb = nullptr; }},
      {"null out", KF_ERR_INVALID_ARG, [](Call& c) { c.out = nullptr; }},
      {"out misaligned to 8", KF_ERR_INVALID_ARG, [](Call& c) { c.out = misalign(c.out, 4); }},
  };
  for (int it = 0; it < iters; ++it) {
    g_device = (int)rnd(0, 7);
    for (const EntryInfo& e : kMutEntries) {
      const bool no_alloc = e.fn == call_step_no_alloc;
      const bool attn = e.fn == call_partial || e.fn == call_subset || e.fn == call_step || no_alloc;
      const bool step = e.fn == call_step || no_alloc;
      const bool append = e.fn == call_append;
      const bool merge = e.fn == call_merge;
      auto run = [&](const Mut& m) {
        Call c = valid_call();
        if (e.uses_ws) attach_workspace(c, c.R);
        const bool shape_mut = m.apply == nullptr || strstr(m.what, "heads") ||
                               strstr(m.what, "group") || strstr(m.what, "num_") ||
                               strstr(m.what, "pages") || strstr(m.what, "page ids") ||
                               strstr(m.what, "head_dim") || strstr(m.what, "page size") ||
                               strstr(m.what, "dtype") || strstr(m.what, "layout") ||
                               strstr(m.what, "scale") || strstr(m.what, "fp8");
        if (merge && shape_mut && !strstr(m.what, "head_dim") && !strstr(m.what, "num_seqs"))
          return;  // the merge takes no shape struct
        if (merge && (strstr(m.what, "k_pool") || strstr(m.what, "v_pool") ||
                      strstr(m.what, "page_ids")))
          return;
        if (m.apply) m.apply(c);
        g_launches = 0;
        int st;
        if (m.apply == nullptr) {
          Call cc = c;
          kf_shape* none = nullptr;
          // every entry point with a shape argument rejects NULL
          if (e.fn == call_partial)
            st = kf_partial_attn(none, cc.q, cc.k, cc.v, nullptr, nullptr, (kf_route*)cc.routes,
                                 cc.R, cc.maxp, (int32_t*)cc.pids, (float*)cc.o, (float*)cc.lse,
                                 cc.ws, cc.wsb, (int32_t*)cc.flags, nullptr);
          else if (e.fn == call_append)
            st = kf_kv_append(none, cc.k, cc.v, nullptr, nullptr, cc.kn, cc.vn,
                              (kf_route*)cc.routes, cc.R, (int32_t*)cc.tail, (int32_t*)cc.pids,
                              (int32_t*)cc.flags, nullptr);
          else if (e.fn == call_step)
            st = kf_decode_step(none, cc.q, cc.k, cc.v, nullptr, nullptr, cc.kn, cc.vn,
                                (kf_route*)cc.routes, cc.R, (int32_t*)cc.tail, cc.maxp,
                                (int32_t*)cc.pids, (int32_t*)cc.srb, (float*)cc.o, (float*)cc.lse,
                                (float*)cc.out, (float*)cc.lse_out, cc.ws, cc.wsb,
                                (int32_t*)cc.flags, nullptr);
          else if (e.fn == call_gather)
            st = kf_debug_gather(none, cc.k, cc.v, (kf_route*)cc.routes, cc.R, 0, cc.maxp,
                                 (int32_t*)cc.pids, 1, cc.o, cc.out, (int32_t*)cc.flags, nullptr);
          else if (e.fn == call_step_no_alloc)
            st = kf_decode_step_no_alloc(none, cc.q, cc.k, cc.v, nullptr, nullptr, cc.kn, cc.vn,
                                         (kf_route*)cc.routes, cc.R, (int32_t*)cc.tail, cc.maxp,
                                         (int32_t*)cc.pids, (int32_t*)cc.srb, (float*)cc.o,
                                         (float*)cc.lse, (float*)cc.out, (float*)cc.lse_out,
                                         (int32_t*)cc.flags, nullptr);
          else if (e.fn == call_subset)
            st = kf_partial_attn_subset(none, cc.q, cc.k, cc.v, nullptr, nullptr,
                                        (kf_route*)cc.routes, cc.R, (int32_t*)cc.list, cc.nlist,
                                        cc.maxp, (int32_t*)cc.pids, (float*)cc.o, (float*)cc.lse,
                                        cc.ws, cc.wsb, (int32_t*)cc.flags, nullptr);
          else
            return;
        } else if (merge && strstr(m.what, "head_dim")) {
          c.s.head_dim = 64;
          st = e.fn(c);
        } else {
          st = e.fn(c);
        }
        CHECK(st == m.expect, "%s with %s -> %d, expected %d", e.name, m.what, st, m.expect);
        CHECK(g_launches == 0, "%s with %s launched %d kernels", e.name, m.what, g_launches);
        g_ws = nullptr;
      };
      for (const Mut& m : muts) {
        if (merge && !strstr(m.what, "null err_flags") && !strstr(m.what, "misaligned err") &&
            !strstr(m.what, "head_dim") && !strstr(m.what, "num_seqs"))
          continue;
        if (e.fn == call_gather && (strstr(m.what, "fp8")))
          continue;  // the gather copies codes and never reads scales
        run(m);
      }
      if (attn)
        for (const Mut& m : attn_muts) {
          if (step && strstr(m.what, "65536")) continue;  // merge grid limit differs; below
          if (no_alloc && strstr(m.what, "workspace")) continue;  // takes no workspace
          run(m);
        }
      if (step || append)
        for (const Mut& m : step_muts) {
          if (append && (strstr(m.what, "seq_route") || strstr(m.what, "out"))) continue;
          run(m);
        }
      // a workspace one block short of what the launch needs
      if (e.fn == call_partial || e.fn == call_step) {
        Call c = valid_call();
        int32_t cp = 0, mc = 0, up = 0;
        if (kf_partial_attn_plan(&c.s, c.R, c.maxp, 0, &cp, &mc, &up) == KF_OK && mc > 1) {
          attach_workspace(c, c.R);
          const size_t need = kf::workspace_layout(c.R, c.s.num_kv_heads,
                                                   c.s.num_q_heads / c.s.num_kv_heads, mc,
                                                   ordered(cp, mc, c.R, c.s.num_kv_heads))
                                  .total;
          c.wsb = need - 256;
          g_launches = 0;
          const int st = e.fn(c);
          CHECK(st == KF_ERR_WORKSPACE && g_launches == 0, "%s short workspace -> %d", e.name, st);
          c.wsb = need;
          g_launches = 0;
          CHECK(e.fn(c) == KF_OK, "%s exact workspace rejected", e.name);
          g_ws = nullptr;
        }
      }
    }
  }
}

// Arbitrary arguments: statuses stay in the documented set; nothing the
// sanitizers can see goes wrong.
static void fuzz(int iters) {
  const int32_t ints[] = {-2147483647 - 1, -65536, -1, 0, 1, 2, 3, 15, 16, 17, 127, 128, 129,
                          255, 256, 65535, 65536, 1 << 20, 2147483647};
  auto any = [&]() -> int32_t {
    return coin(0.5) ? ints[rnd(0, sizeof ints / sizeof ints[0] - 1)] : (int32_t)rnd(-5, 5000);
  };
  auto anyp = [&](int k) -> void* {
    const double u = std::uniform_real_distribution<double>(0, 1)(rng);
    if (u < 0.1) return nullptr;
    if (u < 0.2) return misalign(fake(k), (int)rnd(1, 255));
    return fake(k);
  };
  for (int it = 0; it < iters; ++it) {
    g_device = (int)rnd(0, 7);
    g_no_device = coin(0.05);
    Call c;
    memset(&c, 0, sizeof c);
    c.s.num_seqs = any();
    c.s.num_q_heads = any();
    c.s.num_kv_heads = coin(0.5) ? any() : (int32_t)rnd(1, 16);
    if (coin(0.5) && c.s.num_kv_heads > 0 && c.s.num_kv_heads < 100000)
      c.s.num_q_heads = c.s.num_kv_heads * (int32_t)rnd(1, 17);
    c.s.head_dim = coin(0.8) ? 128 : any();
    c.s.page_size = coin(0.8) ? 16 : any();
    c.s.kv_dtype = coin(0.8) ? (int32_t)rnd(0, 1) : any();
    c.s.num_pages = any();
    c.s.num_page_ids = any();
    const float scales[] = {0.088f, 0.0f, -1.0f, NAN, INFINITY, 1e30f};
    c.s.scale = scales[rnd(0, 5)];
    c.s.kv_layout = coin(0.8) ? (int32_t)rnd(0, 1) : any();
    void** ptrs[] = {&c.q, &c.k, &c.v, &c.ks, &c.vs, &c.kn, &c.vn, &c.routes, &c.tail, &c.pids,
                     &c.srb, &c.o, &c.lse, &c.out, &c.lse_out, &c.flags, &c.list, &c.ws};
    int k = 0;
    for (void** p : ptrs) *p = anyp(++k);
    c.R = any();
    c.maxp = any();
    c.nlist = any();
    c.wsb = coin(0.5) ? (size_t)rnd(0, 1 << 30) : (size_t)-1;
    g_ws = nullptr;
    for (const EntryInfo& e : kMutEntries) {
      const int st = e.fn(c);
      CHECK(known_status(st), "%s fuzz status %d", e.name, st);
      g_ws = nullptr;
    }
    int32_t cp = 0, mc = 0, up = 0;
    const int st = kf_partial_attn_plan(coin(0.05) ? nullptr : &c.s, c.R, c.maxp,
                                        coin(0.9) ? (int32_t)rnd(0, 1) : any(),
                                        coin(0.2) ? nullptr : &cp, coin(0.2) ? nullptr : &mc,
                                        coin(0.2) ? nullptr : &up);
    CHECK(known_status(st), "plan fuzz status %d", st);
    (void)kf_partial_attn_workspace_bytes(coin(0.05) ? nullptr : &c.s, c.R, c.maxp);
    (void)kf_status_str(any());
  }
  g_no_device = false;
}

// Plans of valid launches: ranges cover the longest unit; a workspace of the
// queried size (over num_routes) serves every launch of 1..num_routes routes
// and both readings of the page table; the query stays fast.
static double plans(int iters) {
  double worst_ms = 0;
  for (int it = 0; it < iters; ++it) {
    g_device = (int)rnd(0, 7);
    kf_shape s = valid_shape();
    const int32_t R = (int32_t)(coin(0.2) ? rnd(1, 65535) : rnd(1, 300));
    const int32_t maxp = (int32_t)(coin(0.2) ? rnd(0, 2147483647) : rnd(0, 5000));
    const auto t0 = std::chrono::steady_clock::now();
    const size_t ws = kf_partial_attn_workspace_bytes(&s, R, maxp);
    const double ms =
        std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t0).count();
    if (ms > worst_ms) worst_ms = ms;
    CHECK(ws >= 256, "workspace %zu", ws);
    for (int k = 0; k < 8; ++k) {
      const int32_t m = (int32_t)(k == 0 ? R : rnd(1, R));
      s.num_page_ids = (int32_t)(coin(0.5) ? 0 : ((int64_t)m * maxp > 2147483647 ? 2147483647
                                                                              : (int64_t)m * maxp));
      for (int list = 0; list < 2; ++list) {
        int32_t cp = -1, mc = -1, up = -1;
        const int st = kf_partial_attn_plan(&s, m, maxp, list, &cp, &mc, &up);
        CHECK(st == KF_OK, "plan status %d", st);
        if (st != KF_OK) continue;
        CHECK(cp >= 1 && mc >= 1 && mc <= 65535 && (up == 1 || up == 2), "plan %d %d %d", cp, mc, up);
        CHECK(((int64_t)maxp + cp - 1) / cp <= mc, "plan leaves pages uncovered: %d x %d < %d", mc,
              cp, maxp);
        if (up == 2) CHECK(list == 0 && mc == 1 && s.kv_dtype == KF_KV_BF16, "two-unit mode");
        const size_t need = kf::workspace_layout(m, s.num_kv_heads,
                                                 s.num_q_heads / s.num_kv_heads, mc,
                                                 ordered(cp, mc, m, s.num_kv_heads))
                                .total;
        CHECK(need <= ws, "launch of %d routes needs %zu > queried %zu (R=%d maxp=%d H=%d)", m,
              need, ws, R, maxp, s.num_kv_heads);
      }
    }
  }
  // extremes: the query is bounded for every argument
  const int32_t Rs[] = {65535, 65536, 2147483647, 6144, 1};
  const int32_t Ps[] = {0, 17, 1000, 2147483647};
  for (int dev = 0; dev < 8; ++dev)
    for (int32_t H : {1, 2, 8, 65535, 65536})
      for (int32_t dt : {0, 1})
        for (int32_t R : Rs)
          for (int32_t P : Ps) {
            g_device = dev;
            kf_shape s = valid_shape();
            s.num_kv_heads = H;
            s.num_q_heads = H;
            s.kv_dtype = dt;
            const auto t0 = std::chrono::steady_clock::now();
            const size_t ws = kf_partial_attn_workspace_bytes(&s, R, P);
            const double ms = std::chrono::duration<double, std::milli>(
                                  std::chrono::steady_clock::now() - t0)
                                  .count();
            if (ms > worst_ms) worst_ms = ms;
            if (R > 65535 || H > 65535) CHECK(ws == 0, "query above the launch limit -> %zu", ws);
          }
  return worst_ms;
}

int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 200;
  valid_calls(iters);
  valid_no_alloc(iters * 4);
  one_mutation(iters / 4 + 1);
  fuzz(iters * 20);
  const double worst = plans(iters);
  printf("worst workspace query %.3f ms (sanitized build)\n", worst);
  if (g_errors) {
    printf("api_stress FAILED: %ld errors\n", g_errors);
    return 1;
  }
  printf("api_stress ok\n");
  return 0;
}
