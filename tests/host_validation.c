/*
 * Host-side driver of libacrl's argument validation, built with
 * AddressSanitizer on the host code (tests/test_host_asan.py).  Every call
 * below is out of contract (or a pure host helper), so it returns before any
 * HIP call: no device is needed and none is touched.  Exit status = number of
 * unexpected results.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "acrl.h"

static int failures = 0;

static void expect(const char* what, acrl_status got, acrl_status want) {
  if (got != want) {
    printf("FAIL %s: status %d, expected %d (%s)\n", what, got, want, acrl_last_error());
    ++failures;
  }
}

int main(void) {
  static unsigned char buf[1 << 16] __attribute__((aligned(256)));
  void* p = buf;
  size_t nb = 0;

  /* status strings, version, descriptor sizes (NULL pointers allowed) */
  for (int s = -1; s < 8; ++s)
    if (!acrl_status_string(s) || !acrl_status_string(s)[0]) ++failures;
  if (acrl_abi_version() != ACRL_ABI_VERSION) ++failures;
  size_t sz[6] = {0};
  acrl_abi_struct_sizes(&sz[0], &sz[1], &sz[2], &sz[3], &sz[4], &sz[5]);
  acrl_abi_struct_sizes(NULL, NULL, NULL, NULL, NULL, NULL);
  if (sz[0] != sizeof(acrl_score_desc) || sz[5] != sizeof(acrl_backward_desc)) ++failures;

  /* quantize */
  expect("quantize cols", acrl_quantize_fp8(p, 4, 33, 33, 1, 0, p, p, NULL, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("quantize rows", acrl_quantize_fp8(p, -1, 64, 64, 1, 0, p, p, NULL, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("quantize ld", acrl_quantize_fp8(p, 4, 64, 60, 1, 0, p, p, NULL, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("quantize scaling", acrl_quantize_fp8(p, 4, 64, 64, 9, 0, p, p, NULL, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("quantize rounding", acrl_quantize_fp8(p, 4, 64, 64, 1, 7, p, p, NULL, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("quantize null", acrl_quantize_fp8(NULL, 4, 64, 64, 1, 0, p, p, NULL, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("quantize misaligned", acrl_quantize_fp8(buf + 1, 4, 64, 64, 1, 0, p, p, NULL, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("quantize workspace", acrl_quantize_fp8(p, 4, 64, 64, 0, 0, p, p, NULL, 0, NULL), ACRL_ERR_WORKSPACE);
  expect("quantize huge", acrl_quantize_fp8(p, (int64_t)1 << 40, 64, 64, 1, 0, p, p, NULL, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("quantize ws query", acrl_quantize_workspace_size(4, 64, 0, &nb), ACRL_OK);
  expect("quantize ws null", acrl_quantize_workspace_size(4, 64, 0, NULL), ACRL_ERR_INVALID_ARG);
  expect("encode n", acrl_fp8_encode((const float*)p, -1, 0, p, NULL), ACRL_ERR_INVALID_ARG);
  expect("encode rounding", acrl_fp8_encode((const float*)p, 4, 3, p, NULL), ACRL_ERR_INVALID_ARG);

  /* score */
  acrl_score_desc sd;
  memset(&sd, 0, sizeof sd);
  expect("score null desc", acrl_score_pi_mu(NULL, NULL), ACRL_ERR_INVALID_ARG);
  expect("score zero desc", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  sd.n_rows = 4; sd.d = 256; sd.V = 1000; sd.h = p; sd.w = p; sd.hq = p; sd.hq_scales = p; sd.wq = p;
  sd.wq_scales = p; sd.mu_scaling = 1; sd.inv_temperature = 1.0f; sd.token_ids = (const int32_t*)p;
  sd.logp_pi = (float*)p; sd.logp_mu = (float*)p; sd.workspace = p; sd.workspace_bytes = 16;
  expect("score workspace", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_WORKSPACE);
  sd.workspace_bytes = (size_t)1 << 40;
  sd.d = 100;
  expect("score d", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  sd.d = 256; sd.inv_temperature = -1.0f;
  expect("score tau", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  sd.inv_temperature = 1.0f; sd.div_chunk = -3; sd.l2 = (float*)p;
  expect("score div_chunk", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  sd.div_chunk = 0; sd.V = (int64_t)1 << 40;
  expect("score V", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  sd.V = 1000; sd.l2 = NULL;
  /* policies, packed weights, descriptor workspace query */
  sd.policies = 7;
  expect("score policies", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  sd.policies = ACRL_POLICY_PI; sd.l2 = (float*)p;
  expect("score div one policy", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  sd.l2 = NULL; sd.policies = ACRL_POLICY_MU; sd.hq = NULL;
  expect("score mu hq", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  sd.hq = p; sd.policies = ACRL_POLICY_BOTH; sd.packed_weights = p; sd.packed_weights_bytes = 16;
  expect("score packed bytes", acrl_score_pi_mu(&sd, NULL), ACRL_ERR_INVALID_ARG);
  size_t nb2 = 0, nb3 = 0;
  expect("score ws query desc packed", acrl_score_workspace_query(&sd, &nb2), ACRL_OK);
  sd.packed_weights = NULL;
  expect("score ws query desc", acrl_score_workspace_query(&sd, &nb3), ACRL_OK);
  if (!(nb2 < nb3)) ++failures;
  expect("packed size", acrl_packed_weights_size(1000, 256, 2, &nb2), ACRL_OK);
  expect("packed size d", acrl_packed_weights_size(1000, 100, 2, &nb2), ACRL_ERR_INVALID_ARG);
  expect("pack null", acrl_pack_weights(NULL, p, p, 1000, 256, 1, p, (size_t)1 << 30, NULL), ACRL_ERR_INVALID_ARG);
  expect("pack bytes", acrl_pack_weights(p, p, p, 1000, 256, 1, p, 16, NULL), ACRL_ERR_WORKSPACE);
  expect("score ws query", acrl_score_workspace_size(300, 256, 1000, 1, &nb), ACRL_OK);
  expect("score div ws query", acrl_score_div_workspace_size(300, 256, 1000, 1, 0, &nb), ACRL_OK);
  expect("score ws d", acrl_score_workspace_size(300, 100, 1000, 1, &nb), ACRL_ERR_INVALID_ARG);
  expect("score ws rows x d", acrl_score_workspace_size((int64_t)1 << 30, 1 << 20, 1000, 1, &nb),
         ACRL_ERR_INVALID_ARG);

  /* sampling */
  acrl_sample_desc sp;
  memset(&sp, 0, sizeof sp);
  expect("sample null", acrl_sample_mu(NULL, NULL), ACRL_ERR_INVALID_ARG);
  sp.n_rows = 4; sp.d = 256; sp.V = 1000; sp.hq = p; sp.hq_scales = p; sp.wq = p; sp.wq_scales = p;
  sp.mu_scaling = 0; sp.inv_temperature = 1.0f; sp.ids = (int32_t*)p; sp.row_offset = -1;
  sp.workspace = p; sp.workspace_bytes = (size_t)1 << 40;
  expect("sample row_offset", acrl_sample_mu(&sp, NULL), ACRL_ERR_INVALID_ARG);
  sp.row_offset = 0; sp.workspace_bytes = 1;
  expect("sample workspace", acrl_sample_mu(&sp, NULL), ACRL_ERR_WORKSPACE);

  /* reduce and controller */
  acrl_reduce_desc rd;
  memset(&rd, 0, sizeof rd);
  rd.B = -1; rd.stats = (double*)p;
  expect("reduce B", acrl_discrepancy_reduce(&rd, NULL), ACRL_ERR_INVALID_ARG);
  rd.B = 2; rd.L = 4; rd.n_groups = 1; rd.logp_pi = (float*)p; rd.logp_mu = (float*)p; rd.mask = p;
  rd.group_of_seq = (const int32_t*)p; rd.seq_mean_d = (float*)p; rd.group_y = (float*)p;
  rd.workspace = p; rd.workspace_bytes = 1;
  expect("reduce workspace", acrl_discrepancy_reduce(&rd, NULL), ACRL_ERR_WORKSPACE);
  acrl_controller_desc cd;
  memset(&cd, 0, sizeof cd);
  cd.B = 2; cd.L = 4; cd.n_groups = 1; cd.mask = p; cd.group_of_seq = (const int32_t*)p;
  cd.logp_pi = (float*)p; cd.logp_mu = (float*)p; cd.adv = (float*)p; cd.group_y = (float*)p;
  cd.weight = (float*)p; cd.X = 0.01f; cd.gamma = 0.65f; cd.C = 1.0f;
  expect("controller C", acrl_controller_step(&cd, NULL), ACRL_ERR_INVALID_ARG);
  cd.C = 3.0f; cd.gamma = 0.0f;
  expect("controller gamma", acrl_controller_step(&cd, NULL), ACRL_ERR_INVALID_ARG);
  cd.gamma = 0.65f; cd.X = 0.0f;
  expect("controller X", acrl_controller_step(&cd, NULL), ACRL_ERR_INVALID_ARG);
  cd.X = 0.01f; cd.mode = ACRL_CTRL_MIS;
  expect("controller MIS sums", acrl_controller_step(&cd, NULL), ACRL_ERR_INVALID_ARG);
  cd.mode = ACRL_CTRL_CONTINUOUS; cd.k = 0.0f;
  expect("controller k", acrl_controller_step(&cd, NULL), ACRL_ERR_INVALID_ARG);

  /* surrogate and backward */
  acrl_surrogate_desc su;
  memset(&su, 0, sizeof su);
  su.B = 2; su.L = 4; su.n_groups = 1; su.mask = p; su.group_of_seq = (const int32_t*)p;
  su.logp_new = (float*)p; su.logp_old = (float*)p; su.adv = (float*)p; su.coef = (float*)p;
  su.loss = (double*)p; su.eps_low = 1.0f; su.eps_high = 0.2f;
  expect("surrogate eps", acrl_surrogate(&su, NULL), ACRL_ERR_INVALID_ARG);
  su.eps_low = 0.2f; su.workspace = p; su.workspace_bytes = 1;
  expect("surrogate workspace", acrl_surrogate(&su, NULL), ACRL_ERR_WORKSPACE);
  acrl_backward_desc bd;
  memset(&bd, 0, sizeof bd);
  bd.n_rows = 4; bd.d = 256; bd.V = 1000; bd.h = p; bd.w = p; bd.token_ids = (const int32_t*)p;
  bd.coef = (float*)p; bd.lse = (float*)p; bd.inv_temperature = 1.0f; bd.workspace = p; bd.workspace_bytes = 1;
  expect("backward outputs", acrl_lm_head_backward(&bd, NULL), ACRL_ERR_INVALID_ARG);
  bd.dh = (float*)p;
  expect("backward workspace", acrl_lm_head_backward(&bd, NULL), ACRL_ERR_WORKSPACE);
  bd.V = (int64_t)1 << 23;
  expect("backward V", acrl_lm_head_backward(&bd, NULL), ACRL_ERR_INVALID_ARG);
  expect("backward ws query", acrl_backward_workspace_size(300, 256, 1000, 0, &nb), ACRL_OK);
  expect("backward ws chunk", acrl_backward_workspace_size(300, 256, 1000, -1, &nb), ACRL_ERR_INVALID_ARG);

  /* host helper */
  const float gy[3] = {0.01f, 0.5f, 0.03f};
  const int32_t gn[3] = {8, 0, 8};
  float X = 0.0f;
  expect("reference X", acrl_reference_from_groups(gy, gn, 3, &X), ACRL_OK);
  if (X < 0.0199f || X > 0.0201f) ++failures;
  const int32_t none[3] = {0, 0, 0};
  expect("reference X empty", acrl_reference_from_groups(gy, none, 3, &X), ACRL_ERR_INVALID_ARG);
  expect("reference X null", acrl_reference_from_groups(NULL, gn, 3, &X), ACRL_ERR_INVALID_ARG);

  printf("%d unexpected results\n", failures);
  return failures;
}
