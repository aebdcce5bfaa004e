/* Plain C99 client of libkf: the headers compile as C, and the host entry
 * points (status strings, version, the launch-plan query, the
 * scaling-policy calculator of Section 4.2 on the hand-worked example) run
 * without a GPU. */
#include <math.h>
#include <stdio.h>
#include <string.h>

#include "kf.h"
#include "kf_policy.h"

int main(void) {
  int fails = 0;
  kf_policy_params p;
  memset(&p, 0, sizeof p);
  p.num_kv_heads = 1; p.head_dim = 2; p.num_layers = 1; p.elem_bytes = 2;
  p.beta_mem = 0.5; p.beta_slo = 0.5; p.gamma = 0.9;
  p.t_a_max = 2.0; p.bw_hbm = 30.0; p.c_kv_cap = 200.0; p.t_step = 1.0; p.t_prewarm = 3.0;

  double c = 0, c_mem = 0, c_slo = 0;
  if (kf_policy_threshold(&p, &c, &c_mem, &c_slo) != KF_OK || c != 30.0 || c_mem != 100.0 ||
      c_slo != 30.0) fails |= 1;
  if (kf_policy_token_bytes(&p) != 8) fails |= 2;

  const int64_t lens[3] = {5, 3, 2};
  kf_policy_node nodes[8];
  kf_policy_range ranges[16];
  int32_t tail[3], num_nodes = 0, num_ranges = 0;
  int64_t c_total = 0;
  if (kf_policy_init(&p, lens, 3, 8, 16, &c_total, &num_nodes, nodes, ranges, &num_ranges, tail) !=
      KF_OK || c_total != 80 || num_nodes != 3 || num_ranges != 5) fails |= 4;
  if (ranges[tail[0]].node != 1 || ranges[tail[1]].node != 2 || ranges[tail[2]].node != 2)
    fails |= 8;

  /* a too-small output is refused with the required counts reported */
  int32_t nn = 0, nr = 0;
  if (kf_policy_init(&p, lens, 3, 1, 1, &c_total, &nn, nodes, ranges, &nr, tail) !=
      KF_ERR_CAPACITY || nn != 3 || nr != 5) fails |= 16;

  double exposed = 0, gain = 0;
  if (kf_policy_pipeline(1.0, 2.0, 3.0, &exposed, &gain) != KF_OK || exposed != 3.0 || gain != 2.0)
    fails |= 32;
  if (strcmp(kf_status_str(KF_ERR_WORKSPACE), "workspace missing or too small") != 0) fails |= 64;
  if (strncmp(kf_version(), "kf ", 3) != 0) fails |= 128;
  if (sizeof(kf_route) != 24 || sizeof(kf_policy_params) != 80 || sizeof(kf_policy_node) != 32)
    fails |= 256;

  /* launch plan of the Llama-3.1-8B layer (no GPU: 256 compute units assumed) */
  const kf_shape llama = {16, 32, 8, KF_HEAD_DIM, KF_PAGE_SIZE, KF_KV_BF16, 33000, 33000, 0.0884f,
                          KF_KV_PAGE_MAJOR};
  int32_t chunk_pages = 0, max_chunks = 0, units_per_wg = 0;
  if (kf_partial_attn_plan(&llama, 64, 516, 0, &chunk_pages, &max_chunks, &units_per_wg) != KF_OK ||
      chunk_pages != 516 || max_chunks != 1 || units_per_wg != 2)
    fails |= 512;
  if (kf_partial_attn_plan(&llama, 64, 516, 2, NULL, NULL, NULL) != KF_ERR_INVALID_ARG) fails |= 1024;
  printf("abi_smoke %s (%d)\n", fails ? "FAILED" : "ok", fails);
  return fails ? 1 : 0;
}
