/*
 * kf_policy.h -- C ABI of the attention-node scaling policy: per-node KV
 * budget, post-prefill placement of token ranges, the per-step fill monitor,
 * and the routing table the decode kernels (kf.h) consume.
 *
 * Source: KernelFlume (arXiv 2606.29207), Section 4.2 (Elastic Scaling
 * Policy): Algorithm 1, Eq. (1) (per-node threshold) and Eq. (2) (fill
 * horizon); Section 5.2 (Kernel Pipelining) for the two-stage model that
 * yields the per-layer attention budget.
 *
 * Host code only: every pointer is a HOST pointer owned by the caller, every
 * call is synchronous, nothing is allocated that outlives a call, and no GPU
 * is touched.  Invalid arguments return KF_ERR_INVALID_ARG before any output
 * is written; an output array that is too small returns KF_ERR_CAPACITY
 * with nothing modified (the required counts are reported where stated); a
 * failure to allocate host temporaries returns KF_ERR_HOST_MEMORY (no
 * exception leaves the library).
 *
 * Readings where the paper leaves a choice
 * ----------------------------------------
 *  - bytes per token of one request = 2 (K and V) * H_kv * d_h * L *
 *    elem_bytes (2 in the paper; 1 accepted for 8-bit KV).
 *  - Eq. (1) budgets whole-node bytes over all L layers, while T_A^max is a
 *    per-layer time.  Each layer scans the node's per-layer share C/L at
 *    BW_HBM, so the SLO term in whole-node bytes is
 *    beta_slo * T_A^max * BW_HBM * L (the printed formula when L = 1).
 *  - N_A = max(1, ceil(C_total / C_thresh)).
 *  - Byte-balanced placement: the batch's tokens, request after request, form
 *    one sequence of T tokens and node k owns positions
 *    [floor(k T / N_A), floor((k+1) T / N_A)); a request has one range per
 *    node it overlaps, and its tail is the node of its highest range.  A
 *    request without tokens gets an empty range on the node owning its start
 *    position (the last node when that is T).
 *  - The monitor visits, in increasing id, the nodes that are the tail of at
 *    least one active request.  A prewarm takes the next node id.  Publishing
 *    moves every active tail of the node to the prewarmed node, opening an
 *    empty range there at the request's current length.
 *  - Exact for byte counts below 2^53 (they are compared as doubles).
 */
#ifndef KF_POLICY_H
#define KF_POLICY_H

#include <stdint.h>

#include "kf.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Inputs of Algorithm 1.  Times in seconds, bytes in bytes, bandwidth in
 * bytes per second.  Valid: counts >= 1, elem_bytes 1 or 2, beta_mem,
 * beta_slo and gamma in (0, 1], t_a_max, bw_hbm, c_kv_cap, t_step > 0,
 * t_prewarm >= 0, all finite. */
typedef struct {
  int32_t num_kv_heads; /* H_kv */
  int32_t head_dim;     /* d_h */
  int32_t num_layers;   /* L */
  int32_t elem_bytes;   /* bytes per K or V element */
  double beta_mem;      /* memory headroom factor */
  double beta_slo;      /* SLO headroom factor */
  double gamma;         /* activation watermark (fraction of C_thresh) */
  double t_a_max;       /* largest admissible routed-attention time per layer */
  double bw_hbm;        /* effective HBM bandwidth of one attention node */
  double c_kv_cap;      /* usable KV capacity of one attention node */
  double t_step;        /* predicted decode-step time */
  double t_prewarm;     /* measured time to prepare a new node's route */
} kf_policy_params;

/* Tokens [tok_begin, tok_end) of request `seq` held by node `node`. */
typedef struct {
  int32_t seq;
  int32_t node;
  int64_t tok_begin;
  int64_t tok_end;
} kf_policy_range;

/* Monitor state of one node. */
typedef struct {
  int64_t bytes;         /* b_i: KV bytes held */
  int32_t live;          /* 1 once the node holds routes; 0 while only reserved by a prewarm */
  int32_t prewarm;       /* id of the node prewarmed for this one, -1 if none */
  int32_t prewarm_ready; /* set by the caller when that prewarm has finished */
  int32_t reserved;      /* 0 */
  double tau_fill;       /* Eq. (2) at the last monitor pass, NaN when not evaluated */
} kf_policy_node;

enum { KF_POLICY_SPAWN = 1, KF_POLICY_PUBLISH = 2 };

/* kind SPAWN: node `node` started prewarming node `new_node`;
 * kind PUBLISH: `count` active tails of `node` moved to `new_node`. */
typedef struct {
  int64_t step;
  int32_t kind;
  int32_t node;
  int32_t new_node;
  int32_t count;
} kf_policy_event;

/* KV bytes one request adds per decode token, or -1 for invalid params. */
int64_t kf_policy_token_bytes(const kf_policy_params* p);

/*
 * kf_policy_threshold -- Eq. (1): C_mem = beta_mem * C_kv_cap,
 * C_slo = beta_slo * T_A^max * BW_HBM * L, C_thresh = min(C_mem, C_slo).
 * Any of the three output pointers may be NULL.
 */
int kf_policy_threshold(const kf_policy_params* p, double* c_thresh, double* c_mem,
                        double* c_slo);

/*
 * kf_policy_layer_budget -- per-layer routed-attention budget (Section 4.2):
 * T_A^max = (t_slo - t_overhead) / num_layers.  KF_ERR_INFEASIBLE when that
 * is not positive or the W-side stage t_w_stage (T_p + T_f) exceeds it.
 */
int kf_policy_layer_budget(double t_slo, double t_overhead, int32_t num_layers,
                           double t_w_stage, double* t_a_max);

/*
 * kf_policy_pipeline -- two-stage pipeline model (Section 5.2): exposed
 * per-layer time max(T_p + T_f, T_A) and the pipelined-to-serial throughput
 * ratio (T_p + T_A + T_f) / exposed.  Times >= 0, not all zero.
 */
int kf_policy_pipeline(double t_p, double t_f, double t_a, double* exposed, double* gain);

/*
 * kf_policy_init -- post-prefill initialisation (Algorithm 1, first block):
 * C_total = sum_i seq_lens[i] * token_bytes, N_A nodes, byte-balanced ranges,
 * the tail of each request.
 *  seq_lens [num_seqs] >= 0.
 *  Out: *c_total; *num_nodes = N_A and nodes[0 .. N_A) (bytes = held bytes,
 *  live = 1, prewarm = -1, tau_fill = NaN); *num_ranges and
 *  ranges[0 .. *num_ranges) ordered by (seq, tok_begin); tail[i] = index in
 *  ranges of request i's tail range.  *num_nodes and *num_ranges are written
 *  also when KF_ERR_CAPACITY is returned (at most num_seqs + N_A - 1 ranges).
 *  KF_ERR_UNSUPPORTED when N_A would exceed INT32_MAX.
 */
int kf_policy_init(const kf_policy_params* p, const int64_t* seq_lens, int32_t num_seqs,
                   int32_t max_nodes, int32_t max_ranges, int64_t* c_total,
                   int32_t* num_nodes, kf_policy_node* nodes, kf_policy_range* ranges,
                   int32_t* num_ranges, int32_t* tail);

/*
 * kf_policy_monitor -- one pass of Algorithm 1's per-step loop at a token
 * boundary.  For each node i holding n_i > 0 active tails:
 *   g_i = n_i * token_bytes, tau_i = (C_thresh - b_i) / g_i     (Eq. (2));
 *   if tau_i * t_step < t_prewarm and no prewarm is pending: reserve node
 *     *num_nodes as i's prewarm (live = 0) and emit SPAWN;
 *   if b_i >= gamma * C_thresh and i's prewarm is ready: move every active
 *     tail of i to it (a new empty range at seq_len[r]), mark it live, clear
 *     i's prewarm and emit PUBLISH.
 *  active [num_seqs] (0/1), seq_len [num_seqs] current lengths; tail
 *  [num_seqs] in/out.  nodes/ranges/events grow in place up to their max;
 *  the call needs room for one more node per tail-holding node, one more
 *  range per active request and two events per tail-holding node, and
 *  returns KF_ERR_CAPACITY (nothing modified) otherwise.
 */
int kf_policy_monitor(const kf_policy_params* p, int64_t step, int32_t num_seqs,
                      const uint8_t* active, const int64_t* seq_len, int32_t* tail,
                      kf_policy_node* nodes, int32_t* num_nodes, int32_t max_nodes,
                      kf_policy_range* ranges, int32_t* num_ranges, int32_t max_ranges,
                      kf_policy_event* events, int32_t* num_events, int32_t max_events);

/*
 * kf_policy_simulate -- init, then `steps` decode steps.  At boundary t:
 * a prewarm spawned at boundary t0 becomes ready once
 * (t - t0) * t_step >= t_prewarm; the monitor runs; then every active request
 * appends one token to its tail range (request i is active for steps
 * 0 .. gen_lens[i]-1).
 *  tails_per_step [steps][num_seqs] (may be NULL): node each request's
 *  append used at step t, -1 when inactive.  seq_len_out [num_seqs]: final
 *  lengths.  *max_node_bytes: the largest b_i seen.  Other outputs as for
 *  kf_policy_init / kf_policy_monitor; KF_ERR_CAPACITY when any array fills
 *  up (outputs are then partial).
 */
int kf_policy_simulate(const kf_policy_params* p, const int64_t* seq_lens,
                       const int64_t* gen_lens, int32_t num_seqs, int64_t steps,
                       int32_t max_nodes, int32_t max_ranges, int32_t max_events,
                       int32_t* tails_per_step, kf_policy_node* nodes, int32_t* num_nodes,
                       kf_policy_range* ranges, int32_t* num_ranges, int32_t* tail,
                       kf_policy_event* events, int32_t* num_events, int64_t* seq_len_out,
                       int64_t* max_node_bytes);

/*
 * kf_policy_build_routes -- routing table (kf_route rows, Section 4.1
 * single-GPU form) for the decode kernels from policy ranges: one route per
 * range, grouped by request (CSR seq_route_begin [num_seqs+1]) and ordered
 * by tok_begin (ties keep range order); part = the range's node; page_cap =
 * ceil((tok_end - tok_begin) / page_size) of the range as given (pass final
 * ranges to reserve room for later appends); tok_end = seq_len_now[seq]
 * clamped to the range.  Pages are taken in route order from free_pages
 * (or 0, 1, 2, ... when free_pages is NULL) into page_ids; *num_page_ids =
 * pages used (also written on KF_ERR_CAPACITY).  range_to_route
 * [num_ranges] maps each range to its row.  Token indices must fit int32.
 */
int kf_policy_build_routes(const kf_policy_range* ranges, int32_t num_ranges,
                           int32_t num_seqs, const int64_t* seq_len_now, int32_t page_size,
                           const int32_t* free_pages, int32_t num_free, kf_route* routes,
                           int32_t* seq_route_begin, int32_t* range_to_route,
                           int32_t* page_ids, int32_t max_page_ids, int32_t* num_page_ids);

#ifdef __cplusplus
}
#endif

#endif /* KF_POLICY_H */
