/*
 * Host paths of the C ABI (include/mtdao.h) under AddressSanitizer and
 * UndefinedBehaviorSanitizer, with no GPU: configuration validation, the
 * schedule, workspace and scratch sizes, handle creation over addresses
 * that are never dereferenced (init_states = 1 launches nothing), argument
 * errors of every entry point, the empty problem (numel = 0), error strings
 * and destruction.  Exit status 0 when every call returned what the header
 * promises.
 */
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "mtdao.h"

static int failures = 0;
#define EXPECT(cond)                                                         \
  do {                                                                       \
    if (!(cond)) {                                                           \
      fprintf(stderr, "%s:%d: expectation failed: %s\n", __FILE__, __LINE__, #cond); \
      ++failures;                                                            \
    }                                                                        \
  } while (0)

static mtdao_config base_config(void) {
  mtdao_config c;
  memset(&c, 0, sizeof c);
  c.form = MTDAO_ADAM;
  c.replicas = 4;
  c.n_moments = 2;
  c.beta1[0] = 0.9f;
  c.beta1[1] = 0.99f;
  c.omega[0] = 0.5f;
  c.omega[1] = 0.3f;
  c.beta2 = 0.999f;
  c.eps = 1e-8f;
  c.period_x = 4;
  c.period_u[0] = 8;
  c.period_u[1] = 8;
  c.period_v = 16;
  c.numel = 1024;
  c.bias_correction = 1;
  return c;
}

/* a handle over fake, never-dereferenced 16-byte aligned addresses */
static mtdao_handle* fake_handle(const mtdao_config* c) {
  mtdao_buffers b;
  memset(&b, 0, sizeof b);
  uintptr_t base = (uintptr_t)1 << 40, stride = (uintptr_t)1 << 36;
  b.x = (void*)base;
  for (int j = 0; j < c->n_moments; ++j) b.u[j] = (float*)(base + (uintptr_t)(j + 1) * stride);
  b.v = c->form == MTDAO_SGDM ? NULL : (float*)(base + 5 * stride);
  b.x_outer = (float*)(base + 6 * stride);
  b.x_outer_mom = (float*)(base + 7 * stride);
  b.init_states = 1;
  size_t ws = 0;
  EXPECT(mtdao_workspace_bytes(c, &ws) == MTDAO_OK);
  mtdao_handle* h = NULL;
  int32_t r = mtdao_init(c, &b, ws ? (void*)(base + 8 * stride) : NULL, ws, NULL, &h);
  EXPECT(r == MTDAO_OK && h != NULL);
  return h;
}

int main(void) {
  /* invalid configurations: every one rejected with a message */
  for (int k = 0; k < 14; ++k) {
    mtdao_config c = base_config();
    int64_t tn[3] = {500, 500, 25};
    switch (k) {
      case 0: c.form = 3; break;
      case 1: c.replicas = 0; break;
      case 2: c.n_moments = 5; break;
      case 3: c.beta1[0] = 1.0f; break;
      case 4: c.omega[0] = 0.9f; break; /* sum 1.2 */
      case 5: c.period_x = -1; break;
      case 6: c.eps = -1.0f; break;
      case 7: c.numel = -5; break;
      case 8: c.n_tensors = 3; c.tensor_numel = tn; break; /* sums to 1025 */
      case 9: c.n_tensors = 2; c.tensor_numel = NULL; break;
      case 10: c.form = MTDAO_ADOPT; c.clip_rho = 1.0f; break;
      case 11: c.outer_opt = MTDAO_OUTER_NESTEROV; c.outer_lr = 0.0f; break;
      case 12: c.sync_order = MTDAO_SYNC_MOMENTA_IN_STEP; break; /* Adam */
      default: c.param_dtype = 7; break;
    }
    size_t n = 0;
    EXPECT(mtdao_workspace_bytes(&c, &n) == MTDAO_ERR_INVALID_ARG);
    EXPECT(strlen(mtdao_last_error(NULL)) > 0);
    mtdao_handle* h = (mtdao_handle*)0x1;
    mtdao_buffers b;
    memset(&b, 0, sizeof b);
    EXPECT(mtdao_init(&c, &b, NULL, 0, NULL, &h) == MTDAO_ERR_INVALID_ARG);
  }

  /* the schedule over many steps, sizes of the workspace and scratch */
  mtdao_config c = base_config();
  for (int64_t s = 1; s <= 4096; ++s) {
    uint32_t m = 0;
    EXPECT(mtdao_schedule(&c, s, &m) == MTDAO_OK);
    uint32_t want = (s % 4 == 0 ? 1u : 0u) | (s % 8 == 0 ? 6u : 0u) | (s % 16 == 0 ? 8u : 0u);
    EXPECT(m == want);
  }
  uint32_t m0;
  EXPECT(mtdao_schedule(&c, 0, &m0) == MTDAO_ERR_RANGE);
  size_t ws = 1, ss = 0;
  EXPECT(mtdao_workspace_bytes(&c, &ws) == MTDAO_OK && ws == 0);
  EXPECT(mtdao_stats_scratch_bytes(&c, &ss) == MTDAO_OK && ss > 0);
  mtdao_config clip = base_config();
  clip.form = MTDAO_SGDM;
  clip.clip_rho = 1.0f;
  clip.numel = 1 << 20;
  EXPECT(mtdao_workspace_bytes(&clip, &ws) == MTDAO_OK && ws >= 4 * 256);

  /* init errors with otherwise valid arguments */
  mtdao_buffers b;
  memset(&b, 0, sizeof b);
  mtdao_handle* h = NULL;
  EXPECT(mtdao_init(&c, &b, NULL, 0, NULL, &h) == MTDAO_ERR_INVALID_ARG); /* x NULL */
  b.x = (void*)(uintptr_t)((1ull << 40) + 4);
  b.u[0] = (float*)(uintptr_t)(1ull << 41);
  b.u[1] = (float*)(uintptr_t)(1ull << 42);
  b.v = (float*)(uintptr_t)(1ull << 43);
  b.init_states = 1;
  EXPECT(mtdao_init(&c, &b, NULL, 0, NULL, &h) == MTDAO_ERR_ALIGN);
  b.x = (void*)(uintptr_t)(1ull << 41); /* overlaps u[0] */
  EXPECT(mtdao_init(&c, &b, NULL, 0, NULL, &h) == MTDAO_ERR_INVALID_ARG);
  EXPECT(mtdao_init(&clip, &b, NULL, 0, NULL, &h) != MTDAO_OK);

  /* a handle: argument errors of every call, nothing launched */
  h = fake_handle(&c);
  uint32_t applied = 0;
  EXPECT(mtdao_step_count(h) == 0);
  EXPECT(mtdao_sync(h, 1u << 6, &applied, NULL) == MTDAO_ERR_INVALID_ARG);
  EXPECT(strstr(mtdao_last_error(h), "mask") != NULL);
  EXPECT(mtdao_sync(h, MTDAO_SYNC_AUTO, &applied, NULL) == MTDAO_OK && applied == 0); /* s = 0 */
  EXPECT(mtdao_local_step(h, NULL, 1e-3f, 0.0f, NULL) == MTDAO_ERR_INVALID_ARG);
  EXPECT(mtdao_local_step(h, (void*)(uintptr_t)((1ull << 44) + 8), 1e-3f, 0.0f, NULL) == MTDAO_ERR_ALIGN);
  EXPECT(mtdao_local_step(h, (void*)(uintptr_t)(1ull << 40), 1e-3f, 0.0f, NULL) == MTDAO_ERR_INVALID_ARG);
  float nan = 0.0f / 0.0f;
  EXPECT(mtdao_step_sync(h, (void*)(uintptr_t)(1ull << 44), nan, 0.0f, 0, &applied, NULL) == MTDAO_ERR_INVALID_ARG);
  EXPECT(mtdao_step_count(h) == 0);
  double stats[(MTDAO_MAX_N + 2) * MTDAO_STATS_STRIDE];
  EXPECT(mtdao_sync_stats(h, 1, &applied, NULL, 0, stats, NULL) == MTDAO_ERR_WORKSPACE);
  EXPECT(mtdao_sync_stats(h, 1, &applied, (void*)(uintptr_t)((1ull << 44) + 64), ss, stats, NULL) == MTDAO_ERR_ALIGN);
  EXPECT(mtdao_sync_stats(h, 0, &applied, (void*)(uintptr_t)(1ull << 44), ss, stats, NULL) == MTDAO_OK);
  EXPECT(stats[0] != stats[0]); /* NaN rows: nothing averaged */
  float dst[4];
  EXPECT(mtdao_read_state(h, 9, 0, 0, 4, dst, NULL) == MTDAO_ERR_INVALID_ARG);
  EXPECT(mtdao_read_state(h, 0, 4, 0, 4, dst, NULL) == MTDAO_ERR_RANGE);
  EXPECT(mtdao_read_state(h, 0, 0, 1022, 4, dst, NULL) == MTDAO_ERR_RANGE);
  EXPECT(mtdao_read_state(h, 0, 0, 0, 0, dst, NULL) == MTDAO_OK);
  EXPECT(mtdao_read_state(h, MTDAO_STATE_X_OUTER, 0, 0, 4, dst, NULL) == MTDAO_ERR_INVALID_ARG);
  mtdao_destroy(h);

  /* the empty problem: steps count, masks are reported, nothing launched */
  mtdao_config e = base_config();
  e.numel = 0;
  memset(&b, 0, sizeof b);
  h = NULL;
  EXPECT(mtdao_init(&e, &b, NULL, 0, NULL, &h) == MTDAO_OK);
  for (int s = 1; s <= 32; ++s) {
    EXPECT(mtdao_step_sync(h, NULL, 1e-3f, 0.0f, MTDAO_SYNC_AUTO, &applied, NULL) == MTDAO_OK);
    uint32_t want = 0;
    EXPECT(mtdao_schedule(&e, s, &want) == MTDAO_OK && applied == want);
  }
  EXPECT(mtdao_step_count(h) == 32);
  mtdao_destroy(h);
  mtdao_destroy(NULL);
  EXPECT(mtdao_step_count(NULL) == -1);

  if (failures) {
    fprintf(stderr, "%d expectations failed\n", failures);
    return 1;
  }
  printf("host ABI paths clean under the sanitizers\n");
  return 0;
}
