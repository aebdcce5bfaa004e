// Attention-node scaling policy (KernelFlume, arXiv 2606.29207, Section 4.2:
// Algorithm 1, Eqs. (1) and (2); Section 5.2 pipeline model) and the routing
// table it hands to the decode kernels.  Host code; see kf_policy.h for the
// contract and the readings.
//
// Floating-point expressions are written in one fixed order (left to right,
// byte counts converted to double where they meet a double) so that results
// are reproducible bit for bit.
#include <algorithm>
#include <climits>
#include <cmath>
#include <cstdint>
#include <limits>
#include <vector>

#include "kf_policy.h"

namespace {

bool pos_finite(double x) { return std::isfinite(x) && x > 0.0; }
bool unit_interval(double x) { return std::isfinite(x) && x > 0.0 && x <= 1.0; }

bool valid(const kf_policy_params* p) {
  return p && p->num_kv_heads >= 1 && p->head_dim >= 1 && p->num_layers >= 1 &&
         (p->elem_bytes == 1 || p->elem_bytes == 2) && unit_interval(p->beta_mem) &&
         unit_interval(p->beta_slo) && unit_interval(p->gamma) && pos_finite(p->t_a_max) &&
         pos_finite(p->bw_hbm) && pos_finite(p->c_kv_cap) && pos_finite(p->t_step) &&
         std::isfinite(p->t_prewarm) && p->t_prewarm >= 0.0;
}

int64_t token_bytes(const kf_policy_params* p) {
  return (int64_t)2 * p->num_kv_heads * p->head_dim * p->num_layers * p->elem_bytes;
}

double thresh(const kf_policy_params* p, double* c_mem_out = nullptr, double* c_slo_out = nullptr) {
  const double c_mem = p->beta_mem * p->c_kv_cap;
  const double c_slo = p->beta_slo * p->t_a_max * p->bw_hbm * (double)p->num_layers;
  if (c_mem_out) *c_mem_out = c_mem;
  if (c_slo_out) *c_slo_out = c_slo;
  return c_slo < c_mem ? c_slo : c_mem;
}

// floor(k * T / n) without overflow
int64_t cut_at(int64_t k, int64_t total, int64_t n) {
  return (int64_t)(((__int128)k * total) / n);
}

void fresh_node(kf_policy_node* nd, int64_t bytes, int32_t live) {
  nd->bytes = bytes;
  nd->live = live;
  nd->prewarm = -1;
  nd->prewarm_ready = 0;
  nd->reserved = 0;
  nd->tau_fill = std::numeric_limits<double>::quiet_NaN();
}

// The node whose position interval contains g (the last node for g = T).
int64_t node_of(int64_t g, int64_t total, int64_t n) {
  if (total == 0 || g >= total) return n - 1;
  int64_t k = (int64_t)(((__int128)g * n) / total);
  while (cut_at(k + 1, total, n) <= g) ++k;
  while (k > 0 && cut_at(k, total, n) > g) --k;
  return k;
}

// Post-prefill placement: emit(i, node, tok_begin, tok_end) for every range,
// request by request, nodes in increasing order.
template <class Emit>
void place(const int64_t* lens, int32_t B, int64_t T, int64_t n, Emit emit) {
  int64_t start = 0;
  for (int32_t i = 0; i < B; ++i) {
    const int64_t s = lens[i];
    if (s == 0) {
      emit(i, node_of(start, T, n), 0, 0);
      continue;
    }
    for (int64_t k = node_of(start, T, n); k < n; ++k) {
      const int64_t lo = std::max(cut_at(k, T, n), start);
      const int64_t hi = std::min(cut_at(k + 1, T, n), start + s);
      if (lo >= start + s) break;
      if (lo < hi) emit(i, k, lo - start, hi - start);
    }
    start += s;
  }
}

}  // namespace

extern "C" {

int64_t kf_policy_token_bytes(const kf_policy_params* p) {
  return valid(p) ? token_bytes(p) : -1;
}

int kf_policy_threshold(const kf_policy_params* p, double* c_thresh, double* c_mem,
                        double* c_slo) {
  if (!valid(p)) return KF_ERR_INVALID_ARG;
  const double c = thresh(p, c_mem, c_slo);
  if (c_thresh) *c_thresh = c;
  return KF_OK;
}

int kf_policy_layer_budget(double t_slo, double t_overhead, int32_t num_layers,
                           double t_w_stage, double* t_a_max) {
  if (!t_a_max || num_layers < 1 || !std::isfinite(t_slo) || !std::isfinite(t_overhead) ||
      !std::isfinite(t_w_stage) || t_w_stage < 0.0)
    return KF_ERR_INVALID_ARG;
  const double bud = (t_slo - t_overhead) / (double)num_layers;
  if (bud <= 0.0 || t_w_stage > bud) return KF_ERR_INFEASIBLE;
  *t_a_max = bud;
  return KF_OK;
}

int kf_policy_pipeline(double t_p, double t_f, double t_a, double* exposed, double* gain) {
  if (!exposed || !gain || !std::isfinite(t_p) || !std::isfinite(t_f) || !std::isfinite(t_a) ||
      t_p < 0.0 || t_f < 0.0 || t_a < 0.0)
    return KF_ERR_INVALID_ARG;
  const double w = t_p + t_f;
  const double e = t_a > w ? t_a : w;
  if (!(e > 0.0)) return KF_ERR_INVALID_ARG;
  *exposed = e;
  *gain = (t_p + t_a + t_f) / e;
  return KF_OK;
}

int kf_policy_init(const kf_policy_params* p, const int64_t* seq_lens, int32_t num_seqs,
                   int32_t max_nodes, int32_t max_ranges, int64_t* c_total,
                   int32_t* num_nodes, kf_policy_node* nodes, kf_policy_range* ranges,
                   int32_t* num_ranges, int32_t* tail) {
  if (!valid(p) || num_seqs < 0 || (num_seqs > 0 && (!seq_lens || !tail)) || !c_total ||
      !num_nodes || !num_ranges || max_nodes < 0 || max_ranges < 0)
    return KF_ERR_INVALID_ARG;
  int64_t T = 0;
  for (int32_t i = 0; i < num_seqs; ++i) {
    if (seq_lens[i] < 0) return KF_ERR_INVALID_ARG;
    if (seq_lens[i] > INT64_MAX - T) return KF_ERR_UNSUPPORTED;
    T += seq_lens[i];
  }
  const int64_t tb = token_bytes(p);
  if (T > 0 && T > INT64_MAX / tb) return KF_ERR_UNSUPPORTED;
  const int64_t total_bytes = T * tb;
  const double need = std::ceil((double)total_bytes / thresh(p));
  if (need > (double)INT32_MAX) return KF_ERR_UNSUPPORTED;
  const int64_t n = std::max<int64_t>(1, (int64_t)need);
  int64_t nr = 0;
  place(seq_lens, num_seqs, T, n, [&](int32_t, int64_t, int64_t, int64_t) { ++nr; });
  *c_total = total_bytes;
  *num_nodes = (int32_t)n;
  *num_ranges = (int32_t)std::min<int64_t>(nr, INT32_MAX);
  if (n > max_nodes || nr > max_ranges || !nodes || (nr > 0 && !ranges)) return KF_ERR_CAPACITY;

  for (int64_t k = 0; k < n; ++k) fresh_node(&nodes[k], 0, 1);
  int32_t w = 0;
  place(seq_lens, num_seqs, T, n, [&](int32_t i, int64_t k, int64_t b, int64_t e) {
    ranges[w] = kf_policy_range{i, (int32_t)k, b, e};
    nodes[k].bytes += (e - b) * tb;
    tail[i] = w++;  // the last range emitted for request i is its highest
  });
  return KF_OK;
}

static int kf_policy_monitor_impl(const kf_policy_params* p, int64_t step, int32_t num_seqs,
                      const uint8_t* active, const int64_t* seq_len, int32_t* tail,
                      kf_policy_node* nodes, int32_t* num_nodes, int32_t max_nodes,
                      kf_policy_range* ranges, int32_t* num_ranges, int32_t max_ranges,
                      kf_policy_event* events, int32_t* num_events, int32_t max_events) {
  if (!valid(p) || num_seqs < 0 || !nodes || !num_nodes || !ranges || !num_ranges ||
      !num_events || (max_events > 0 && !events) ||
      (num_seqs > 0 && (!active || !seq_len || !tail)))
    return KF_ERR_INVALID_ARG;
  const int32_t N = *num_nodes;
  int32_t R = *num_ranges;
  if (N < 0 || N > max_nodes || R < 0 || R > max_ranges || *num_events < 0 ||
      *num_events > max_events)
    return KF_ERR_INVALID_ARG;
  for (int32_t r = 0; r < num_seqs; ++r) {
    if (!active[r]) continue;
    if (tail[r] < 0 || tail[r] >= R) return KF_ERR_INVALID_ARG;
    const int32_t nd = ranges[tail[r]].node;
    if (nd < 0 || nd >= N) return KF_ERR_INVALID_ARG;
  }
  for (int32_t i = 0; i < N; ++i)
    if (nodes[i].prewarm >= N || nodes[i].prewarm < -1) return KF_ERR_INVALID_ARG;

  // active tails per node, bucketed by node in request order
  std::vector<int32_t> cnt(N + 1, 0);
  int32_t n_active = 0;
  for (int32_t r = 0; r < num_seqs; ++r)
    if (active[r]) {
      ++cnt[ranges[tail[r]].node + 1];
      ++n_active;
    }
  int32_t holders = 0;
  for (int32_t i = 0; i < N; ++i) holders += cnt[i + 1] > 0;
  if ((int64_t)N + holders > max_nodes || (int64_t)R + n_active > max_ranges ||
      (int64_t)*num_events + 2 * holders > max_events)
    return KF_ERR_CAPACITY;
  for (int32_t i = 0; i < N; ++i) cnt[i + 1] += cnt[i];
  std::vector<int32_t> order(n_active);
  {
    std::vector<int32_t> fill(cnt.begin(), cnt.end() - 1);
    for (int32_t r = 0; r < num_seqs; ++r)
      if (active[r]) order[fill[ranges[tail[r]].node]++] = r;
  }

  const double c_thresh = thresh(p);
  const int64_t tb = token_bytes(p);
  int32_t nn = N, ne = *num_events;
  for (int32_t i = 0; i < N; ++i) nodes[i].tau_fill = std::numeric_limits<double>::quiet_NaN();
  for (int32_t i = 0; i < N; ++i) {
    const int32_t n_i = cnt[i + 1] - cnt[i];
    if (n_i == 0) continue;
    kf_policy_node& nd = nodes[i];
    const int64_t g_i = (int64_t)n_i * tb;
    const int64_t b_i = nd.bytes;
    const double tau = (c_thresh - (double)b_i) / (double)g_i;
    nd.tau_fill = tau;
    if (tau * p->t_step < p->t_prewarm && nd.prewarm < 0) {
      fresh_node(&nodes[nn], 0, 0);
      nd.prewarm = nn++;
      nd.prewarm_ready = 0;
      events[ne++] = kf_policy_event{step, KF_POLICY_SPAWN, i, nd.prewarm, 0};
    }
    if ((double)b_i >= p->gamma * c_thresh && nd.prewarm >= 0 && nd.prewarm_ready) {
      const int32_t j = nd.prewarm;
      for (int32_t k = cnt[i]; k < cnt[i + 1]; ++k) {
        const int32_t r = order[k];
        ranges[R] = kf_policy_range{r, j, seq_len[r], seq_len[r]};
        tail[r] = R++;
      }
      nodes[j].live = 1;
      nd.prewarm = -1;
      nd.prewarm_ready = 0;
      events[ne++] = kf_policy_event{step, KF_POLICY_PUBLISH, i, j, n_i};
    }
  }
  *num_nodes = nn;
  *num_ranges = R;
  *num_events = ne;
  return KF_OK;
}

static int kf_policy_simulate_impl(const kf_policy_params* p, const int64_t* seq_lens,
                       const int64_t* gen_lens, int32_t num_seqs, int64_t steps,
                       int32_t max_nodes, int32_t max_ranges, int32_t max_events,
                       int32_t* tails_per_step, kf_policy_node* nodes, int32_t* num_nodes,
                       kf_policy_range* ranges, int32_t* num_ranges, int32_t* tail,
                       kf_policy_event* events, int32_t* num_events, int64_t* seq_len_out,
                       int64_t* max_node_bytes) {
  if (!valid(p) || num_seqs < 0 || steps < 0 || !num_events || !max_node_bytes ||
      (num_seqs > 0 && (!gen_lens || !seq_len_out)))
    return KF_ERR_INVALID_ARG;
  for (int32_t i = 0; i < num_seqs; ++i)
    if (gen_lens[i] < 0) return KF_ERR_INVALID_ARG;
  int64_t c_total = 0;
  int st = kf_policy_init(p, seq_lens, num_seqs, max_nodes, max_ranges, &c_total, num_nodes,
                          nodes, ranges, num_ranges, tail);
  if (st != KF_OK) return st;
  *num_events = 0;
  const int64_t tb = token_bytes(p);
  std::vector<int64_t> left(gen_lens, gen_lens + num_seqs);
  std::vector<uint8_t> active(num_seqs);
  for (int32_t i = 0; i < num_seqs; ++i) {
    active[i] = left[i] > 0;
    seq_len_out[i] = seq_lens[i];
  }
  std::vector<int64_t> spawned_at(max_nodes, -1);
  int64_t peak = 0;
  for (int32_t k = 0; k < *num_nodes; ++k) peak = std::max(peak, nodes[k].bytes);
  for (int64_t t = 0; t < steps; ++t) {
    for (int32_t k = 0; k < *num_nodes; ++k) {
      const int32_t j = nodes[k].prewarm;
      if (j >= 0 && !nodes[k].prewarm_ready &&
          (double)(t - spawned_at[j]) * p->t_step >= p->t_prewarm)
        nodes[k].prewarm_ready = 1;
    }
    const int32_t ev0 = *num_events;
    st = kf_policy_monitor(p, t, num_seqs, active.data(), seq_len_out, tail, nodes, num_nodes,
                           max_nodes, ranges, num_ranges, max_ranges, events, num_events,
                           max_events);
    if (st != KF_OK) return st;
    for (int32_t e = ev0; e < *num_events; ++e)
      if (events[e].kind == KF_POLICY_SPAWN) spawned_at[events[e].new_node] = t;
    for (int32_t i = 0; i < num_seqs; ++i) {
      int32_t* row = tails_per_step ? tails_per_step + t * num_seqs : nullptr;
      if (!active[i]) {
        if (row) row[i] = -1;
        continue;
      }
      kf_policy_range& rg = ranges[tail[i]];
      if (row) row[i] = rg.node;
      rg.tok_end += 1;
      nodes[rg.node].bytes += tb;
      seq_len_out[i] += 1;
      if (--left[i] == 0) active[i] = 0;
    }
    for (int32_t k = 0; k < *num_nodes; ++k) peak = std::max(peak, nodes[k].bytes);
  }
  *max_node_bytes = peak;
  return KF_OK;
}

static int kf_policy_build_routes_impl(const kf_policy_range* ranges, int32_t num_ranges,
                           int32_t num_seqs, const int64_t* seq_len_now, int32_t page_size,
                           const int32_t* free_pages, int32_t num_free, kf_route* routes,
                           int32_t* seq_route_begin, int32_t* range_to_route,
                           int32_t* page_ids, int32_t max_page_ids, int32_t* num_page_ids) {
  if (num_ranges < 0 || num_seqs < 0 || page_size < 1 || !seq_route_begin || !num_page_ids ||
      (num_ranges > 0 && (!ranges || !routes || !range_to_route)) ||
      (num_seqs > 0 && !seq_len_now) || max_page_ids < 0 || (free_pages && num_free < 0))
    return KF_ERR_INVALID_ARG;
  int64_t pages = 0;
  for (int32_t k = 0; k < num_ranges; ++k) {
    const kf_policy_range& g = ranges[k];
    if (g.seq < 0 || g.seq >= num_seqs || g.tok_begin < 0 || g.tok_end < g.tok_begin ||
        g.tok_end > INT32_MAX || g.node < 0)
      return KF_ERR_INVALID_ARG;
    pages += (g.tok_end - g.tok_begin + page_size - 1) / page_size;
  }
  if (pages > INT32_MAX) return KF_ERR_UNSUPPORTED;
  *num_page_ids = (int32_t)pages;
  if (pages > max_page_ids || (pages > 0 && !page_ids) || (free_pages && pages > num_free))
    return KF_ERR_CAPACITY;

  std::vector<int32_t> order(num_ranges);
  for (int32_t k = 0; k < num_ranges; ++k) order[k] = k;
  std::stable_sort(order.begin(), order.end(), [&](int32_t a, int32_t b) {
    if (ranges[a].seq != ranges[b].seq) return ranges[a].seq < ranges[b].seq;
    return ranges[a].tok_begin < ranges[b].tok_begin;
  });
  for (int32_t i = 0; i <= num_seqs; ++i) seq_route_begin[i] = 0;
  int32_t base = 0;
  for (int32_t row = 0; row < num_ranges; ++row) {
    const int32_t k = order[row];
    const kf_policy_range& g = ranges[k];
    const int32_t cap = (int32_t)((g.tok_end - g.tok_begin + page_size - 1) / page_size);
    const int64_t now = std::max(g.tok_begin, std::min(g.tok_end, seq_len_now[g.seq]));
    routes[row] = kf_route{g.seq, g.node, (int32_t)g.tok_begin, (int32_t)now, base, cap};
    range_to_route[k] = row;
    for (int32_t q = 0; q < cap; ++q) page_ids[base + q] = free_pages ? free_pages[base + q] : base + q;
    base += cap;
    ++seq_route_begin[g.seq + 1];
  }
  for (int32_t i = 0; i < num_seqs; ++i) seq_route_begin[i + 1] += seq_route_begin[i];
  return KF_OK;
}

int kf_policy_monitor(const kf_policy_params* p, int64_t step, int32_t num_seqs,
                      const uint8_t* active, const int64_t* seq_len, int32_t* tail,
                      kf_policy_node* nodes, int32_t* num_nodes, int32_t max_nodes,
                      kf_policy_range* ranges, int32_t* num_ranges, int32_t max_ranges,
                      kf_policy_event* events, int32_t* num_events, int32_t max_events) {
  try {
    return kf_policy_monitor_impl(p, step, num_seqs, active, seq_len, tail, nodes, num_nodes, max_nodes, ranges, num_ranges, max_ranges, events, num_events, max_events);
  } catch (...) {  // host temporaries could not be allocated: no exception crosses the C ABI
    return KF_ERR_HOST_MEMORY;
  }
}

int kf_policy_simulate(const kf_policy_params* p, const int64_t* seq_lens,
                       const int64_t* gen_lens, int32_t num_seqs, int64_t steps,
                       int32_t max_nodes, int32_t max_ranges, int32_t max_events,
                       int32_t* tails_per_step, kf_policy_node* nodes, int32_t* num_nodes,
                       kf_policy_range* ranges, int32_t* num_ranges, int32_t* tail,
                       kf_policy_event* events, int32_t* num_events, int64_t* seq_len_out,
                       int64_t* max_node_bytes) {
  try {
    return kf_policy_simulate_impl(p, seq_lens, gen_lens, num_seqs, steps, max_nodes, max_ranges, max_events, tails_per_step, nodes, num_nodes, ranges, num_ranges, tail, events, num_events, seq_len_out, max_node_bytes);
  } catch (...) {  // host temporaries could not be allocated: no exception crosses the C ABI
    return KF_ERR_HOST_MEMORY;
  }
}

int kf_policy_build_routes(const kf_policy_range* ranges, int32_t num_ranges,
                           int32_t num_seqs, const int64_t* seq_len_now, int32_t page_size,
                           const int32_t* free_pages, int32_t num_free, kf_route* routes,
                           int32_t* seq_route_begin, int32_t* range_to_route,
                           int32_t* page_ids, int32_t max_page_ids, int32_t* num_page_ids) {
  try {
    return kf_policy_build_routes_impl(ranges, num_ranges, num_seqs, seq_len_now, page_size, free_pages, num_free, routes, seq_route_begin, range_to_route, page_ids, max_page_ids, num_page_ids);
  } catch (...) {  // host temporaries could not be allocated: no exception crosses the C ABI
    return KF_ERR_HOST_MEMORY;
  }
}

}  // extern "C"
