/*
 * kf.h -- C ABI of the weightless attention node's decode hot path on MI355X
 * (gfx950): tail append, local partial attention over token-range routes,
 * and the log-sum-exp merge of partials.
 *
 * Source: KernelFlume (arXiv 2606.29207).  Section 3.2 (Workflow of Elastic
 * Decoding), steps 3 and 4; Section 4.1 (Elastic Communication: the routing
 * table from token ranges to the nodes that hold them, one live tail per
 * request); Section 5.1 (Query-First Attention: the tail appends before it
 * attends, and the merge of partials equals attention over the whole range).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - All array pointers are DEVICE pointers owned by the caller; shape
 *    structs are host pointers.  The library allocates and frees nothing.
 *  - Every call is asynchronous on `stream` (a hipStream_t; NULL = the null
 *    stream) and returns once its kernels are enqueued.
 *  - Host-checkable problems (null pointers, misalignment, unsupported
 *    shapes, a workspace that is too small) return a negative status before
 *    anything is launched.
 *  - Problems only the device can see (inconsistent route rows, page ids
 *    outside the pool, a full tail) OR a KF_EFLAG_* bit into *err_flags (a
 *    device int32 the caller zeroes and reads after synchronising).  Outputs
 *    of an affected route or sequence are NaN; an append that fails leaves the
 *    pools and the route unchanged.  Nothing is ever read or written outside
 *    the arrays described here.
 *  - Calls that share buffers must be ordered on one stream: within a decode
 *    step, kf_kv_append -> kf_partial_attn -> kf_merge_partials.
 *
 * Storage formats
 * ---------------
 *  page    = 16 consecutive tokens of one route; head_dim = 128.
 *  K pool  [num_pages][num_kv_heads][16 slots][128] elements (token-major)
 *  V pool  [num_pages][num_kv_heads][128][16 slots] elements (dim-major)
 *            shape->kv_layout = KF_KV_HEAD_MAJOR swaps the two outer
 *            dimensions of both pools: [num_kv_heads][num_pages][...].
 *  element = bfloat16 (KF_KV_BF16) or OCP E4M3FN code (KF_KV_FP8_E4M3);
 *            fp8 pools carry k_scale/v_scale [num_pages][num_kv_heads] float32
 *            and an element's value is decode(code) * scale.
 *  q       [num_seqs][num_q_heads][128] bfloat16; query head h reads KV head
 *            h / (num_q_heads / num_kv_heads).
 *  route r covers logical tokens [tok_begin, tok_end) of sequence `seq`;
 *            local index j = t - tok_begin lives in page
 *            page_ids[page_base + j / 16], slot j % 16.  Routes must not share
 *            pages.  Routes of sequence b are rows
 *            seq_route_begin[b] .. seq_route_begin[b+1]-1.
 */
#ifndef KF_H
#define KF_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define KF_PAGE_SIZE 16
#define KF_HEAD_DIM 128
#define KF_MAX_GROUP 16 /* num_q_heads / num_kv_heads may not exceed this */

/* One entry of the routing table (Section 4.1), single-GPU form: a token
 * range of one request and the pages that hold it.  `part` names the
 * partition (attention node) that owns the range; kernels do not read it. */
typedef struct {
  int32_t seq;       /* sequence index in [0, num_seqs) */
  int32_t part;      /* owning partition id (informational) */
  int32_t tok_begin; /* first logical token of the range */
  int32_t tok_end;   /* one past the last resident token; the tail grows it */
  int32_t page_base; /* index in page_ids of the range's first page */
  int32_t page_cap;  /* pages reserved: page_ids[page_base .. page_base+page_cap) */
} kf_route;

typedef struct {
  int32_t num_seqs;     /* B */
  int32_t num_q_heads;  /* Hq, a multiple of num_kv_heads */
  int32_t num_kv_heads; /* Hkv */
  int32_t head_dim;     /* must be KF_HEAD_DIM */
  int32_t page_size;    /* must be KF_PAGE_SIZE */
  int32_t kv_dtype;     /* KF_KV_BF16 or KF_KV_FP8_E4M3 */
  int32_t num_pages;    /* pages in each of the K and V pools (>= 1) */
  int32_t num_page_ids; /* entries of page_ids */
  float scale;          /* softmax scale applied to q.k, e.g. 1/sqrt(128) */
  int32_t kv_layout;    /* KF_KV_PAGE_MAJOR (0, the default) or KF_KV_HEAD_MAJOR */
} kf_shape;

/* Pool layouts.  Page-major keeps a page's KV heads together; head-major
 * keeps each KV head's pages together.  Results are identical.  Measured on
 * one MI355X over 2.15 GB layers (4.3 GB fp8): head-major streamed 2% faster
 * with 2 KV heads (bf16 and fp8), the same with 4 or 16, and 2% slower with 8.
 * The scales of fp8 pools are [num_pages][num_kv_heads] in both. */
enum { KF_KV_PAGE_MAJOR = 0, KF_KV_HEAD_MAJOR = 1 };

enum {
  KF_OK = 0,
  KF_ERR_INVALID_ARG = -1, /* null/misaligned pointer or inconsistent sizes */
  KF_ERR_UNSUPPORTED = -2, /* a shape or dtype the library does not handle */
  KF_ERR_WORKSPACE = -3,   /* workspace missing or smaller than required */
  KF_ERR_HIP = -4,         /* the HIP runtime refused a launch */
  KF_ERR_CAPACITY = -5,    /* a caller-sized host output array is too small */
  KF_ERR_INFEASIBLE = -6,  /* no budget satisfies the constraints */
  KF_ERR_HOST_MEMORY = -7, /* host-side temporaries could not be allocated */
  KF_ERR_SCRATCH_LIMIT = -8 /* the launch needs more than KF_SCRATCH_BYTES of scratch */
};

/* Size of the library's per-device scratch array (kf_decode_step_no_alloc). */
#define KF_SCRATCH_BYTES ((size_t)32 << 20)

enum { KF_KV_BF16 = 0, KF_KV_FP8_E4M3 = 1 };

enum {
  KF_EFLAG_TAIL_FULL = 1, /* tail has no reserved page for the new token */
  KF_EFLAG_BAD_ROUTE = 2, /* route row / tail index / CSR row inconsistent */
  KF_EFLAG_BAD_PAGE = 4   /* a page id lies outside [0, num_pages) */
};

/*
 * kf_kv_append -- tail append (Section 3.2, step 3; Section 5.1).
 * For every sequence b with r = tail_route[b] >= 0: write k_new[b][g][:] and
 * v_new[b][g][:] (bfloat16 [num_seqs][num_kv_heads][128]) for all KV heads g
 * at local index j = routes[r].tok_end - routes[r].tok_begin of route r, then
 * set routes[r].tok_end += 1.  tail_route[b] = -1 marks a sequence without
 * an append this step.  Device checks (flag, no write): r < num_routes,
 * routes[r].seq == b, tok_end >= tok_begin, j/16 < page_cap
 * (KF_EFLAG_TAIL_FULL otherwise), page_base + j/16 < num_page_ids, page id in
 * the pool.
 * bf16 pools: the token's bits are copied; k_scale/v_scale may be NULL.
 * fp8 pools (the paper has no fp8 KV; this is the library's rule), per page
 * and KV head, separately for K and V, in float32: the first token of a page
 * sets scale = amax/28 (1 if amax = 0), i.e. 16x headroom below 448; a later
 * token whose amax exceeds 448*scale first re-encodes the page's earlier
 * slots to scale' = amax/28 (code' = RNE(decode(code)*scale/scale')); the
 * token is stored as the E4M3 code nearest to x/scale (ties to even, clamped
 * to +-448).
 * Alignment: every pointer 4-byte aligned.
 */
int kf_kv_append(const kf_shape* shape, void* k_pool, void* v_pool, float* k_scale,
                 float* v_scale, const void* k_new, const void* v_new, kf_route* routes,
                 int32_t num_routes, const int32_t* tail_route, const int32_t* page_ids,
                 int32_t* err_flags, void* stream);

/*
 * kf_partial_attn_workspace_bytes -- device scratch kf_partial_attn needs for
 * `num_routes` routes of at most `max_pages_per_route` pages each on the
 * current device (at least 256 bytes).  One workgroup handles a whole
 * (route, KV head) unit when the units fill the GPU evenly; otherwise each
 * unit is split over several workgroups whose partials go through this
 * workspace; a split launch of at least two rounds of resident
 * workgroups also keeps its dispatch order there (8 bytes per work item, a
 * table that a one-workgroup kernel writes before the partial kernel).  The
 * size covers every launch of at most `num_routes` routes, so a workspace
 * sized for a route table also serves
 * kf_partial_attn_subset over any part of it, and it covers ragged and
 * equal routes alike: it does not depend on shape->num_page_ids, so it stays
 * valid as the page table grows or shrinks.  No initialisation is needed;
 * contents are dead between calls.  Returns 0 for invalid arguments and for
 * num_routes or num_kv_heads above 65535, which no launch accepts.  Host
 * only; its time is bounded for any argument (well under a millisecond).
 */
size_t kf_partial_attn_workspace_bytes(const kf_shape* shape, int32_t num_routes,
                                       int32_t max_pages_per_route);

/*
 * kf_partial_attn_plan -- how a partial-attention launch of `num_launch`
 * routes of at most `max_pages_per_route` pages runs on the current device:
 * kf_partial_attn and kf_decode_step (route_list_launch = 0), or
 * kf_partial_attn_subset over a list of num_launch routes
 * (route_list_launch = 1).  Not an operation of the paper: a description of
 * this implementation's launch, for callers that size or inspect it.
 *   *chunk_pages  pages per workgroup range; a unit of n pages is cut into
 *                 ceil(n / chunk_pages) ranges
 *   *max_chunks   most ranges per unit; 1 = every unit whole, no combine
 *                 launch and no workspace use.  A split launch whose
 *                 max_chunks * num_kv_heads * num_launch work items reach
 *                 two per resident workgroup slot (two slots per compute
 *                 unit) and stay within 2^20 is dispatched largest ranges
 *                 first, in an order a one-workgroup kernel computes
 *   *units_per_wg 1 or 2 (route, KV head) units per workgroup
 * The plan reads the launch size, the KV heads and dtype, the device's
 * compute units, max_pages_per_route and shape->num_page_ids: a page table
 * under 90% of num_launch * max_pages_per_route marks the routes as ragged,
 * and ragged routes are cut into more ranges.  Equal units stay whole when
 * they fill whole rounds of two per compute unit or spread evenly over the
 * compute units (units mod CUs is 0 or at least 3/4 of the CUs); other
 * equal units take the fewest ranges (up to 16) that give at least two work
 * items per compute unit, spread evenly so.  Launches over a route list
 * (route_list_launch = 1) skip these two rules: the page table does not
 * tell whether a list's routes are equal.  A max_pages_per_route far
 * above the longest route therefore costs speed, never correctness.
 * Host only; launches nothing.  Any output pointer may be NULL.  Returns
 * KF_OK, KF_ERR_INVALID_ARG (null or invalid shape, negative sizes,
 * route_list_launch not 0 or 1) or KF_ERR_UNSUPPORTED (a shape or size the
 * kernels do not take, as kf_partial_attn would report).
 */
int kf_partial_attn_plan(const kf_shape* shape, int32_t num_launch, int32_t max_pages_per_route,
                         int32_t route_list_launch, int32_t* chunk_pages, int32_t* max_chunks,
                         int32_t* units_per_wg);

/*
 * kf_partial_attn -- local core attention of every route (Section 3.2,
 * step 3): for route r of sequence b and query head h,
 *   s_t = scale * (q[b][h] . k_t) over the route's resident tokens t,
 *   o_part[r][h][:] = sum_t softmax(s)_t v_t     (float32, normalised)
 *   lse_part[r][h]  = ln sum_t exp(s_t)          (float32, natural log)
 * An empty route (tok_end == tok_begin) gives o = 0, lse = -inf.
 * Device checks (NaN outputs + KF_EFLAG_BAD_ROUTE): 0 <= seq < num_seqs,
 * tok_end >= tok_begin, page_base >= 0, pages <= page_cap,
 * pages <= max_pages_per_route, page_base + pages <= num_page_ids; a page id
 * outside the pool gives NaN + KF_EFLAG_BAD_PAGE.
 * k_scale/v_scale: NULL for bf16 pools, required for fp8 pools.
 * o_part [num_routes][num_q_heads][128], lse_part [num_routes][num_q_heads].
 * Alignment: q, pools and o_part 16-byte aligned; the rest 4-byte aligned;
 * workspace 256-byte aligned.
 */
int kf_partial_attn(const kf_shape* shape, const void* q, const void* k_pool,
                    const void* v_pool, const float* k_scale, const float* v_scale,
                    const kf_route* routes, int32_t num_routes,
                    int32_t max_pages_per_route, const int32_t* page_ids,
                    float* o_part, float* lse_part, void* workspace,
                    size_t workspace_bytes, int32_t* err_flags, void* stream);

/*
 * kf_partial_attn_subset -- kf_partial_attn restricted to the routes listed
 * in route_list[0 .. num_list) (device int32 indices into routes[]); other
 * rows of o_part/lse_part are left untouched.  With it the step can be
 * scheduled query-first (Section 5.1): the partials of routes that hold only
 * historical tokens need nothing but q and can start before the step's new
 * K/V token exists, while the tail routes append and then attend on another
 * stream.  Size the workspace with kf_partial_attn_workspace_bytes(shape,
 * num_list, max_pages_per_route) (any larger count also fits); calls that may
 * run concurrently need separate workspaces.  A list entry outside [0, num_routes) sets
 * KF_EFLAG_BAD_ROUTE and writes nothing.  Other arguments, checks and
 * alignment as for kf_partial_attn (route_list 4-byte aligned).
 */
int kf_partial_attn_subset(const kf_shape* shape, const void* q, const void* k_pool,
                           const void* v_pool, const float* k_scale, const float* v_scale,
                           const kf_route* routes, int32_t num_routes,
                           const int32_t* route_list, int32_t num_list,
                           int32_t max_pages_per_route, const int32_t* page_ids,
                           float* o_part, float* lse_part, void* workspace,
                           size_t workspace_bytes, int32_t* err_flags, void* stream);

/*
 * kf_merge_partials -- log-sum-exp merge of the partials of each sequence
 * (Section 3.2, step 4): over the routes r of sequence b,
 *   M = max_r lse_r,  w_r = exp(lse_r - M),
 *   out[b][h][:] = sum_r w_r o_part[r][h][:] / sum_r w_r,
 *   lse_out[b][h] = M + ln sum_r w_r.
 * A sequence with no routes, or only empty ones, gives out = 0, lse = -inf.
 * A CSR row outside [0, num_routes] or decreasing gives NaN +
 * KF_EFLAG_BAD_ROUTE.  out [num_seqs][num_q_heads][head_dim] float32,
 * lse_out [num_seqs][num_q_heads]; head_dim must be KF_HEAD_DIM.
 * Alignment: o_part and out 8-byte aligned; the rest 4-byte aligned.
 */
int kf_merge_partials(int32_t num_seqs, int32_t num_routes, int32_t num_q_heads,
                      int32_t head_dim, const float* o_part, const float* lse_part,
                      const int32_t* seq_route_begin, float* out, float* lse_out,
                      int32_t* err_flags, void* stream);

/*
 * kf_decode_step -- one whole decode step (Section 3.2, steps 3 and 4;
 * Section 5.1): the tail append, partial attention of every route and the
 * merge, with the results, flags and route updates of
 *   kf_kv_append -> kf_partial_attn -> kf_merge_partials
 * on the same arguments (each argument as documented there; the workspace
 * is sized by kf_partial_attn_workspace_bytes), in two launches instead of
 * three (a split launch adds its combine and, over several rounds, its
 * dispatch order, as kf_partial_attn does): the workgroup that attends over
 * a tail's last page first writes the step's token into it (for fp8 pools
 * by the E4M3 append rule, re-encoding the page if needed) and attends over
 * it, and the merge advances the tails' tok_end and raises the append's
 * flags.  All host checks of the three calls
 * are made before anything is launched.
 */
int kf_decode_step(const kf_shape* shape, const void* q, void* k_pool, void* v_pool,
                   float* k_scale, float* v_scale, const void* k_new, const void* v_new,
                   kf_route* routes, int32_t num_routes, const int32_t* tail_route,
                   int32_t max_pages_per_route, const int32_t* page_ids,
                   const int32_t* seq_route_begin, float* o_part, float* lse_part, float* out,
                   float* lse_out, void* workspace, size_t workspace_bytes, int32_t* err_flags,
                   void* stream);

/*
 * kf_decode_step_no_alloc -- kf_decode_step for callers that cannot allocate
 * device memory or pass a workspace: code under HIP graph capture, tight
 * serving loops, harnesses that forbid hipMalloc.  Same arguments, results,
 * flags and route updates as kf_decode_step, without workspace and
 * workspace_bytes: the chunk partials of a split launch go through a scratch
 * array of KF_SCRATCH_BYTES that the library holds in each device's memory
 * from the first kernel launch on that device until the process ends.
 * Allocates nothing and calls no allocating routine.  The first call on a
 * device also looks up that device's array address (hipGetSymbolAddress, on
 * the current device, which must be the stream's); make one call before
 * capturing a graph of it.
 * Returns KF_ERR_SCRATCH_LIMIT, before anything is launched, when the launch
 * would need more scratch than KF_SCRATCH_BYTES: the size kf_partial_attn
 * would require of its workspace for these routes (with 256 compute units,
 * about 4 MiB per query head of a KV group when the (route, KV head) units
 * outnumber two per compute unit without filling whole rounds; launches
 * whose units are not split need none).
 * All calls on one device share its array and nothing in it needs to start
 * at zero; calls that may overlap on one device (streams not ordered with
 * respect to each other) race on it and must be serialised by the caller.
 */
int kf_decode_step_no_alloc(const kf_shape* shape, const void* q, void* k_pool, void* v_pool,
                            float* k_scale, float* v_scale, const void* k_new,
                            const void* v_new, kf_route* routes, int32_t num_routes,
                            const int32_t* tail_route, int32_t max_pages_per_route,
                            const int32_t* page_ids, const int32_t* seq_route_begin,
                            float* o_part, float* lse_part, float* out, float* lse_out,
                            int32_t* err_flags, void* stream);

/*
 * kf_debug_gather -- test export: the resident tokens of route `route`
 * gathered through the routing table by the same route checks and page
 * lookup the attention kernels use (Section 4.1, one route = one token range
 * and the pages that hold it).  With n = min(tok_end - tok_begin,
 * max_tokens), token j < n of the route sits in page
 * page_ids[page_base + j / 16], slot j % 16, and out_k[j][g][:],
 * out_v[j][g][:] receive its K and V elements for every KV head g (bf16 bits,
 * or E4M3 codes for fp8 pools; scales are not applied).  Rows j >= n are not
 * written.  A route row failing kf_partial_attn's checks sets
 * KF_EFLAG_BAD_ROUTE and writes nothing; a page id outside the pool sets
 * KF_EFLAG_BAD_PAGE and leaves that page's rows unwritten.  route must lie in
 * [0, num_routes) (else KF_ERR_INVALID_ARG).  out_k/out_v: device
 * [max_tokens][num_kv_heads][128] elements.  Alignment: 4 bytes.
 */
int kf_debug_gather(const kf_shape* shape, const void* k_pool, const void* v_pool,
                    const kf_route* routes, int32_t num_routes, int32_t route,
                    int32_t max_pages_per_route, const int32_t* page_ids, int32_t max_tokens,
                    void* out_k, void* out_v, int32_t* err_flags, void* stream);

/* Static description of a status code (never NULL). */
const char* kf_status_str(int status);

/* Library build string, e.g. "kf 0.1 gfx950". */
const char* kf_version(void);

#ifdef __cplusplus
}
#endif

#endif /* KF_H */
