/* Memory-safety stress of the scaling-policy host code (include/kf_policy.h),
 * built with AddressSanitizer and UndefinedBehaviorSanitizer by
 * tests/test_host_sanitizers.py.  Every output array is heap-allocated at
 * exactly the capacity passed to the library, so a write past a stated
 * capacity is reported.  Random batches and parameters come from a fixed
 * linear congruential generator; the values themselves are checked against
 * the oracle elsewhere, here only status codes and bounds are. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "kf.h"
#include "kf_policy.h"

static unsigned long long g_state = 0x9E3779B97F4A7C15ull;

static unsigned rnd(unsigned n) { /* uniform-ish in [0, n) */
  g_state = g_state * 6364136223846793005ull + 1442695040888963407ull;
  return n ? (unsigned)((g_state >> 33) % n) : 0u;
}

static double urand(void) { return (double)rnd(1u << 30) / (double)(1u << 30); }

static void* xmalloc(size_t n) {
  void* p = malloc(n ? n : 1);
  if (!p) {
    fprintf(stderr, "out of memory\n");
    exit(2);
  }
  return p;
}

static int fails = 0;
static long long g_spawns = 0, g_publishes = 0, g_refusals = 0;
#define CHECK(cond)                                                  \
  do {                                                               \
    if (!(cond)) {                                                   \
      fprintf(stderr, "check failed line %d: %s\n", __LINE__, #cond); \
      ++fails;                                                       \
    }                                                                \
  } while (0)

static kf_policy_params random_params(void) {
  kf_policy_params p;
  memset(&p, 0, sizeof p);
  p.num_kv_heads = 1 + (int32_t)rnd(2);
  p.head_dim = 1 + (int32_t)rnd(4);
  p.num_layers = 1 + (int32_t)rnd(3);
  p.elem_bytes = 1 + (int32_t)rnd(2);
  p.beta_mem = 0.1 + 0.9 * urand();
  p.beta_slo = 0.1 + 0.9 * urand();
  p.gamma = 0.05 + 0.95 * urand();
  p.t_a_max = 0.5 + 4.0 * urand();
  p.bw_hbm = 50.0 + 5000.0 * urand();
  p.c_kv_cap = 500.0 + 50000.0 * urand();
  p.t_step = 0.5 + urand();
  p.t_prewarm = 5.0 * urand();
  return p;
}

static void scalar_calls(void) {
  kf_policy_params p = random_params();
  double c = 0, cm = 0, cs = 0;
  CHECK(kf_policy_threshold(&p, &c, &cm, &cs) == KF_OK);
  CHECK(kf_policy_threshold(&p, NULL, NULL, NULL) == KF_OK);
  CHECK(kf_policy_token_bytes(&p) > 0);
  kf_policy_params bad = p;
  bad.beta_mem = NAN;
  CHECK(kf_policy_threshold(&bad, &c, &cm, &cs) == KF_ERR_INVALID_ARG);
  CHECK(kf_policy_token_bytes(&bad) == -1);
  bad = p;
  bad.num_layers = 0;
  CHECK(kf_policy_threshold(&bad, &c, &cm, &cs) == KF_ERR_INVALID_ARG);
  CHECK(kf_policy_threshold(NULL, &c, &cm, &cs) == KF_ERR_INVALID_ARG);
  double t = 0, e = 0, gain = 0;
  const int st = kf_policy_layer_budget(50.0, 5.0 * urand(), 1 + (int32_t)rnd(40), 2.0 * urand(), &t);
  CHECK(st == KF_OK || st == KF_ERR_INFEASIBLE);
  CHECK(kf_policy_layer_budget(1.0, 2.0, 4, 0.0, &t) == KF_ERR_INFEASIBLE);
  CHECK(kf_policy_pipeline(urand(), urand(), urand() + 0.01, &e, &gain) == KF_OK);
  CHECK(kf_policy_pipeline(0.0, 0.0, 0.0, &e, &gain) == KF_ERR_INVALID_ARG);
}

static void one_batch(void) {
  kf_policy_params p = random_params();
  const int32_t B = (int32_t)rnd(24);
  int64_t* lens = xmalloc(sizeof(int64_t) * (size_t)B);
  int64_t* gen = xmalloc(sizeof(int64_t) * (size_t)B);
  for (int32_t i = 0; i < B; ++i) {
    lens[i] = rnd(6) == 0 ? 0 : (int64_t)rnd(3000);
    gen[i] = (int64_t)rnd(120);
  }

  /* init: sizes first (no room: refused, counts reported), then exact buffers */
  int64_t c_total = 0;
  int32_t nn = 0, nr = 0;
  int32_t* tail = xmalloc(sizeof(int32_t) * (size_t)B);
  int st = kf_policy_init(&p, lens, B, 0, 0, &c_total, &nn, NULL, NULL, &nr, tail);
  CHECK(st == KF_ERR_CAPACITY || st == KF_ERR_UNSUPPORTED);
  if (st != KF_ERR_CAPACITY || nn > 100000) goto done;
  {
    const int32_t extra_nodes = 2 * B + 4, extra_ranges = 4 * B + 4;
    const int32_t max_nodes = nn + extra_nodes, max_ranges = nr + extra_ranges;
    const int32_t max_events = 4 * (nn + extra_nodes);
    kf_policy_node* nodes = xmalloc(sizeof(kf_policy_node) * (size_t)max_nodes);
    kf_policy_range* ranges = xmalloc(sizeof(kf_policy_range) * (size_t)max_ranges);
    kf_policy_event* events = xmalloc(sizeof(kf_policy_event) * (size_t)max_events);
    /* exactly nn nodes and nr ranges */
    kf_policy_node* nodes_x = xmalloc(sizeof(kf_policy_node) * (size_t)nn);
    kf_policy_range* ranges_x = xmalloc(sizeof(kf_policy_range) * (size_t)nr);
    int32_t n2 = 0, r2 = 0;
    CHECK(kf_policy_init(&p, lens, B, nn, nr, &c_total, &n2, nodes_x, ranges_x, &r2, tail) ==
          KF_OK);
    CHECK(n2 == nn && r2 == nr);
    free(nodes_x);
    free(ranges_x);
    if (nn > 1) { /* one node short: refused */
      kf_policy_node* small = xmalloc(sizeof(kf_policy_node) * (size_t)(nn - 1));
      kf_policy_range* rs = xmalloc(sizeof(kf_policy_range) * (size_t)nr);
      CHECK(kf_policy_init(&p, lens, B, nn - 1, nr, &c_total, &n2, small, rs, &r2, tail) ==
            KF_ERR_CAPACITY);
      free(small);
      free(rs);
    }
    int32_t num_nodes = 0, num_ranges = 0, num_events = 0;
    CHECK(kf_policy_init(&p, lens, B, max_nodes, max_ranges, &c_total, &num_nodes, nodes, ranges,
                         &num_ranges, tail) == KF_OK);

    /* monitor passes with growing lengths; capacity refusals on the way */
    uint8_t* active = xmalloc((size_t)B);
    int64_t* cur = xmalloc(sizeof(int64_t) * (size_t)B);
    for (int32_t i = 0; i < B; ++i) {
      active[i] = (uint8_t)(rnd(4) != 0);
      cur[i] = lens[i];
    }
    for (int64_t step = 0; step < 40; ++step) {
      const int32_t cap_n = rnd(8) == 0 ? num_nodes : max_nodes;
      st = kf_policy_monitor(&p, step, B, active, cur, tail, nodes, &num_nodes, cap_n, ranges,
                             &num_ranges, max_ranges, events, &num_events, max_events);
      CHECK(st == KF_OK || st == KF_ERR_CAPACITY);
      if (st == KF_ERR_CAPACITY) ++g_refusals;
      if (st == KF_ERR_CAPACITY && cap_n == max_nodes) break; /* arrays full */
      for (int32_t i = 0; i < num_nodes; ++i)
        if (nodes[i].prewarm >= 0 && rnd(2)) nodes[i].prewarm_ready = 1;
      for (int32_t i = 0; i < B; ++i) {
        if (!active[i]) continue;
        cur[i] += 1;
        kf_policy_range* r = &ranges[tail[i]];
        r->tok_end += 1;
        nodes[r->node].bytes += kf_policy_token_bytes(&p);
      }
    }

    for (int32_t i = 0; i < num_events; ++i) {
      g_spawns += events[i].kind == KF_POLICY_SPAWN;
      g_publishes += events[i].kind == KF_POLICY_PUBLISH;
    }

    /* routing table for the kernels from the final ranges */
    int32_t* srb = xmalloc(sizeof(int32_t) * (size_t)(B + 1));
    kf_route* routes = xmalloc(sizeof(kf_route) * (size_t)(num_ranges ? num_ranges : 1));
    int32_t* r2r = xmalloc(sizeof(int32_t) * (size_t)(num_ranges ? num_ranges : 1));
    int32_t npid = 0;
    st = kf_policy_build_routes(ranges, num_ranges, B, cur, 16, NULL, 0, routes, srb, r2r, NULL, 0,
                                &npid);
    CHECK(st == KF_OK || st == KF_ERR_CAPACITY);
    int32_t* pids = xmalloc(sizeof(int32_t) * (size_t)(npid ? npid : 1));
    int32_t* free_pages = xmalloc(sizeof(int32_t) * (size_t)(npid ? npid : 1));
    for (int32_t i = 0; i < npid; ++i) free_pages[i] = npid - 1 - i;
    int32_t used = 0;
    CHECK(kf_policy_build_routes(ranges, num_ranges, B, cur, 16, NULL, 0, routes, srb, r2r, pids,
                                 npid, &used) == KF_OK);
    CHECK(used == npid);
    CHECK(kf_policy_build_routes(ranges, num_ranges, B, cur, 16, free_pages, npid, routes, srb, r2r,
                                 pids, npid, &used) == KF_OK);
    if (npid > 0)
      CHECK(kf_policy_build_routes(ranges, num_ranges, B, cur, 16, free_pages, npid - 1, routes,
                                   srb, r2r, pids, npid, &used) == KF_ERR_CAPACITY);
    free(pids);
    free(free_pages);
    free(srb);
    free(routes);
    free(r2r);
    free(active);
    free(cur);

    /* whole simulation, with room and without */
    const int64_t steps = (int64_t)rnd(150);
    int32_t* tps = xmalloc(sizeof(int32_t) * (size_t)(steps * B + 1));
    int64_t* out_len = xmalloc(sizeof(int64_t) * (size_t)(B ? B : 1));
    int64_t max_b = 0;
    st = kf_policy_simulate(&p, lens, gen, B, steps, max_nodes, max_ranges, max_events, tps, nodes,
                            &num_nodes, ranges, &num_ranges, tail, events, &num_events, out_len,
                            &max_b);
    CHECK(st == KF_OK || st == KF_ERR_CAPACITY);
    st = kf_policy_simulate(&p, lens, gen, B, steps, nn, nr, 1, NULL, nodes, &num_nodes, ranges,
                            &num_ranges, tail, events, &num_events, out_len, &max_b);
    CHECK(st == KF_OK || st == KF_ERR_CAPACITY);
    free(tps);
    free(out_len);
    free(nodes);
    free(ranges);
    free(events);
  }
done:
  free(tail);
  free(lens);
  free(gen);
}

int main(int argc, char** argv) {
  const int iters = argc > 1 ? atoi(argv[1]) : 300;
  for (int it = 0; it < iters; ++it) {
    scalar_calls();
    one_batch();
  }
  if (fails) {
    fprintf(stderr, "policy_stress: %d failed checks\n", fails);
    return 1;
  }
  printf("policy_stress ok (%d iterations; monitor: %lld spawns, %lld publishes, %lld refusals)\n",
         iters, g_spawns, g_publishes, g_refusals);
  /* the batches must drive the monitor through both of its actions */
  if (g_spawns == 0 || g_publishes == 0 || g_refusals == 0) return 1;
  return 0;
}
