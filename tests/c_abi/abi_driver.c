/*
 * Plain-C consumer of the MT-DAO C ABI (include/mtdao.h): no Python, no
 * torch.  Device memory comes from hipMalloc, work goes on a HIP stream the
 * program creates, and every state read back through mtdao_read_state is
 * compared with the CPU oracle (oracle/_liboracle.so, test infrastructure)
 * run on the same inputs:
 *   case 1: Adam form (Algorithm 1), N = 3, K = 4 workers, P = 10007 (a
 *           row length that is not a multiple of 4: the scalar path), with
 *           every averaging event folded into mtdao_step_sync;
 *   case 2: SGDM form (Algorithm 3), N = 2, K = 5, P = 8204, per-worker
 *           global-norm clip rho = 0.05 (active), mtdao_local_step followed
 *           by mtdao_sync on the schedule;
 *   case 3: Adam form, N = 2, K = 6, P = 4099, then mtdao_sync_stats of
 *           every state: the averaging diagnostics (Section 4.1's metrics,
 *           in the header's MTDAO_STAT_* layout) against the oracle's on
 *           the same pre-average states, within 1e-5 of
 *           max(|want|, 1e-6 * the largest statistic of the state).
 *   case 4: Adam form with bias correction, N = 2, K = 3, P = 4100, through
 *           a HIP graph: one window of 8 mtdao_step_sync_device calls (the
 *           update number kept on the device, eta_t from a device table that
 *           changes every step) and its mtdao_device_step_advance, captured
 *           once and replayed 3 times, with new gradients written between
 *           replays; the oracle runs the same 24 updates.
 * Every step's mask is also checked against mtdao_schedule (host only).
 * Inputs are seeded splitmix64 fields made here; the driver holds none of
 * the method's arithmetic.  Pass: every applied mask equals the oracle's
 * schedule bit for bit, and every state's max |a - b| / max(|b|, rms(b))
 * is at most 1e-5.  Prints one line per case; exit status 0 on success.
 */
#include <hip/hip_runtime_api.h>
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

#include "mtdao.h"

/* ---- the oracle's C interface (oracle/mtdao_oracle.c) ---- */
typedef struct {
  int32_t form, n, x_dtype, g_dtype, m_dtype, bias_correction, adopt_order;
  float beta1[4], omega[4], beta2, eps;
} oracle_cfg;
uint32_t oracle_schedule(int64_t s, int32_t n, int32_t period_x, const int32_t* period_u, int32_t period_v,
                         int32_t has_v);
double oracle_sumsq(const void* g, int32_t g_dtype, int64_t n);
double oracle_clip_scale(double norm, double rho);
void oracle_local_step(const oracle_cfg* c, int64_t s, float lr, float clip_c, const double* scale, void* x,
                       void* const* u, void* v, const void* g, int64_t K, int64_t P);
void oracle_replica_mean(void* state, int32_t dtype, int64_t K, int64_t P);
void oracle_state_stats(const void* s, int32_t dtype, const float* xo, int64_t K, int64_t P, double* out);

#define CHECK_HIP(call)                                                              \
  do {                                                                               \
    hipError_t e_ = (call);                                                          \
    if (e_ != hipSuccess) {                                                          \
      fprintf(stderr, "%s:%d %s: %s\n", __FILE__, __LINE__, #call, hipGetErrorString(e_)); \
      exit(2);                                                                       \
    }                                                                                \
  } while (0)
#define CHECK_MT(h, call)                                                            \
  do {                                                                               \
    int32_t r_ = (call);                                                             \
    if (r_ != MTDAO_OK) {                                                            \
      fprintf(stderr, "%s:%d %s = %d: %s\n", __FILE__, __LINE__, #call, r_, mtdao_last_error(h)); \
      exit(3);                                                                       \
    }                                                                                \
  } while (0)

/* seeded inputs: splitmix64 -> uniform in [-1, 1) */
static uint64_t mix(uint64_t z) {
  z += 0x9E3779B97F4A7C15ull;
  z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
  z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
  return z ^ (z >> 31);
}
static float field(uint64_t seed, int64_t i) {
  return (float)((double)(mix(seed * 0x100000001B3ull + (uint64_t)i) >> 11) * 0x1p-52 - 1.0);
}

typedef struct {
  const char* name;
  int32_t form, K, N;
  int64_t P;
  float beta1[4], omega[4], beta2, eps, rho, lr;
  int32_t period_x, period_u[4], period_v, steps, fused, stats;
  int32_t graph; /* > 0: steps run as steps / graph replays of a captured window of this many calls */
} drv_case;

/* eta_t of the graph case: a ramp, so that every update takes its own value */
static float ramp_lr(float lr, int64_t s) { return lr * (1.0f + 0.05f * (float)s); }

static double compare(const float* a, const float* b, int64_t n) {
  double ss = 0.0, worst = 0.0;
  for (int64_t i = 0; i < n; ++i) ss += (double)b[i] * (double)b[i];
  const double rms = sqrt(ss / (double)(n > 0 ? n : 1));
  for (int64_t i = 0; i < n; ++i) {
    const double den = fmax(fabs((double)b[i]), rms);
    const double d = den > 0.0 ? fabs((double)a[i] - (double)b[i]) / den : fabs((double)a[i] - (double)b[i]);
    if (!(d <= worst)) worst = d; /* NaN propagates as a failure */
  }
  return worst;
}

static int run_case(const drv_case* t) {
  const int32_t K = t->K, N = t->N;
  const int64_t P = t->P, KP = (int64_t)K * P;
  const int has_v = t->form != MTDAO_SGDM;
  hipStream_t st;
  CHECK_HIP(hipStreamCreate(&st));

  mtdao_config c;
  memset(&c, 0, sizeof c);
  c.form = t->form;
  c.replicas = K;
  c.n_moments = N;
  c.param_dtype = MTDAO_F32;
  c.grad_dtype = MTDAO_F32;
  c.adopt_order = MTDAO_ADOPT_PREV;
  c.bias_correction = t->form == MTDAO_ADAM;
  for (int j = 0; j < N; ++j) {
    c.beta1[j] = t->beta1[j];
    c.omega[j] = t->omega[j];
    c.period_u[j] = t->period_u[j];
  }
  c.beta2 = t->beta2;
  c.eps = t->eps;
  c.clip_rho = t->rho;
  c.period_x = t->period_x;
  c.period_v = t->period_v;
  c.numel = P;
  c.sync_order = MTDAO_SYNC_AFTER_STEP;
  c.outer_opt = MTDAO_OUTER_AVERAGE;

  /* device buffers */
  void* dx;
  float* du[MTDAO_MAX_N] = {0};
  float* dv = NULL;
  float* dg;
  void* ws = NULL;
  CHECK_HIP(hipMalloc(&dx, (size_t)KP * 4));
  for (int j = 0; j < N; ++j) CHECK_HIP(hipMalloc((void**)&du[j], (size_t)KP * 4));
  if (has_v) CHECK_HIP(hipMalloc((void**)&dv, (size_t)KP * 4));
  CHECK_HIP(hipMalloc((void**)&dg, (size_t)KP * 4));
  size_t ws_bytes = 0;
  CHECK_MT(NULL, mtdao_workspace_bytes(&c, &ws_bytes));
  if (ws_bytes) CHECK_HIP(hipMalloc(&ws, ws_bytes));

  /* host oracle states and the inputs */
  float* x = malloc((size_t)KP * 4);
  float* u[MTDAO_MAX_N] = {0};
  for (int j = 0; j < N; ++j) u[j] = calloc((size_t)KP, 4);
  float* v = has_v ? calloc((size_t)KP, 4) : NULL;
  float* g = malloc((size_t)KP * 4);
  float* back = malloc((size_t)KP * 4);
  for (int64_t i = 0; i < P; ++i) x[i] = 0.02f * field(7, i);
  for (int32_t m = 1; m < K; ++m) memcpy(x + (int64_t)m * P, x, (size_t)P * 4);
  CHECK_HIP(hipMemcpy(dx, x, (size_t)P * 4, hipMemcpyHostToDevice)); /* row 0: x_0, broadcast by init */

  mtdao_buffers b;
  memset(&b, 0, sizeof b);
  b.x = dx;
  for (int j = 0; j < N; ++j) b.u[j] = du[j];
  b.v = dv;
  b.init_states = 0;
  mtdao_handle* h = NULL;
  CHECK_MT(NULL, mtdao_init(&c, &b, ws, ws_bytes, (void*)st, &h));

  oracle_cfg oc;
  memset(&oc, 0, sizeof oc);
  oc.form = t->form;
  oc.n = N;
  oc.x_dtype = oc.g_dtype = oc.m_dtype = 0; /* fp32 storage */
  oc.bias_correction = c.bias_correction;
  oc.adopt_order = 0;
  for (int j = 0; j < N; ++j) {
    oc.beta1[j] = t->beta1[j];
    oc.omega[j] = t->omega[j];
  }
  oc.beta2 = t->beta2;
  oc.eps = t->eps;
  void* ou[MTDAO_MAX_N];
  for (int j = 0; j < N; ++j) ou[j] = u[j];
  double scale[64];
  int masks_ok = 1;
  uint32_t nsync = 0;

  /* graph case: capture one window, replay it; the oracle runs every update */
  hipGraphExec_t gexec = NULL;
  hipGraph_t graph = NULL;
  mtdao_device_step* dstep = NULL;
  float* dlr = NULL;
  uint32_t captured[64];
  const int32_t W = t->graph;
  const int64_t table_len = 64;
  if (W > 0) {
    float lr_host[64];
    for (int64_t i = 0; i < table_len; ++i) lr_host[i] = ramp_lr(t->lr, i + 1);
    CHECK_HIP(hipMalloc((void**)&dstep, sizeof(mtdao_device_step)));
    CHECK_HIP(hipMalloc((void**)&dlr, (size_t)table_len * 4));
    CHECK_HIP(hipMemcpy(dlr, lr_host, (size_t)table_len * 4, hipMemcpyHostToDevice));
    CHECK_MT(h, mtdao_device_step_set(h, dstep, 0, (void*)st));
    CHECK_HIP(hipStreamSynchronize(st));
    CHECK_HIP(hipStreamBeginCapture(st, hipStreamCaptureModeGlobal));
    for (int32_t k = 0; k < W; ++k)
      CHECK_MT(h, mtdao_step_sync_device(h, dg, dstep, dlr, NULL, table_len, MTDAO_SYNC_AUTO, &captured[k], (void*)st));
    CHECK_MT(h, mtdao_device_step_advance(h, dstep, (void*)st));
    CHECK_HIP(hipStreamEndCapture(st, &graph));
    CHECK_HIP(hipGraphInstantiate(&gexec, graph, NULL, NULL, 0));
  }

  for (int32_t s = 1; s <= t->steps; ++s) {
    if (W > 0) {
      /* one gradient per window, written between replays */
      const int32_t win = (s - 1) / W, k = (s - 1) % W;
      for (int32_t m = 0; m < K; ++m)
        for (int64_t i = 0; i < P; ++i) g[(int64_t)m * P + i] = 1e-2f * field(5000 + 131 * (uint64_t)win + m, i);
      if (k == 0) {
        CHECK_HIP(hipMemcpyAsync(dg, g, (size_t)KP * 4, hipMemcpyHostToDevice, st));
        CHECK_HIP(hipGraphLaunch(gexec, st));
        CHECK_HIP(hipStreamSynchronize(st));
      }
      oracle_local_step(&oc, s, ramp_lr(t->lr, s), 0.0f, NULL, x, ou, v, g, K, P);
      const uint32_t want = oracle_schedule(s, N, t->period_x, t->period_u, t->period_v, has_v);
      if (want & 1u) oracle_replica_mean(x, 0, K, P);
      for (int j = 0; j < N; ++j)
        if (want & (1u << (j + 1))) oracle_replica_mean(u[j], 0, K, P);
      if (has_v && (want & (1u << (N + 1)))) oracle_replica_mean(v, 0, K, P);
      if (captured[k] != want) {
        fprintf(stderr, "%s: step %d captured mask 0x%x, oracle 0x%x\n", t->name, s, captured[k], want);
        masks_ok = 0;
      }
      nsync += (uint32_t)__builtin_popcount(want);
      continue;
    }
    for (int32_t m = 0; m < K; ++m)
      for (int64_t i = 0; i < P; ++i) g[(int64_t)m * P + i] = 1e-2f * field(1000 + 131 * (uint64_t)s + m, i);
    CHECK_HIP(hipMemcpyAsync(dg, g, (size_t)KP * 4, hipMemcpyHostToDevice, st));
    uint32_t applied = 0;
    if (t->fused) {
      CHECK_MT(h, mtdao_step_sync(h, dg, t->lr, 0.0f, MTDAO_SYNC_AUTO, &applied, (void*)st));
    } else {
      CHECK_MT(h, mtdao_local_step(h, dg, t->lr, 0.0f, (void*)st));
      CHECK_MT(h, mtdao_sync(h, MTDAO_SYNC_AUTO, &applied, (void*)st));
    }
    /* the oracle: clip factors, the step, then the schedule's means */
    for (int32_t m = 0; m < K; ++m)
      scale[m] = oracle_clip_scale(sqrt(oracle_sumsq(g + (int64_t)m * P, 0, P)), (double)t->rho);
    oracle_local_step(&oc, s, t->lr, 0.0f, t->rho > 0.0f ? scale : NULL, x, ou, v, g, K, P);
    const uint32_t want = oracle_schedule(s, N, t->period_x, t->period_u, t->period_v, has_v);
    uint32_t sched = 0;
    CHECK_MT(NULL, mtdao_schedule(&c, s, &sched));
    if (sched != want) {
      fprintf(stderr, "%s: step %d mtdao_schedule 0x%x, oracle 0x%x\n", t->name, s, sched, want);
      masks_ok = 0;
    }
    if (want & 1u) oracle_replica_mean(x, 0, K, P);
    for (int j = 0; j < N; ++j)
      if (want & (1u << (j + 1))) oracle_replica_mean(u[j], 0, K, P);
    if (has_v && (want & (1u << (N + 1)))) oracle_replica_mean(v, 0, K, P);
    if (applied != want) {
      fprintf(stderr, "%s: step %d applied mask 0x%x, oracle 0x%x\n", t->name, s, applied, want);
      masks_ok = 0;
    }
    nsync += (uint32_t)__builtin_popcount(want);
    CHECK_HIP(hipStreamSynchronize(st)); /* g is rewritten next step */
  }

  /* every state averaged with its diagnostics */
  const int nstates = 1 + N + (has_v ? 1 : 0);
  double stats_worst = 0.0;
  if (t->stats) {
    size_t sb = 0;
    CHECK_MT(NULL, mtdao_stats_scratch_bytes(&c, &sb));
    void* scratch = NULL;
    CHECK_HIP(hipMalloc(&scratch, sb));
    double hs[(MTDAO_MAX_N + 2) * MTDAO_STATS_STRIDE];
    const uint32_t full = (1u << nstates) - 1u;
    uint32_t applied = 0;
    CHECK_MT(h, mtdao_sync_stats(h, full, &applied, scratch, sb, hs, (void*)st));
    if (applied != full) masks_ok = 0;
    double* want = malloc((size_t)(4 + 2 * K) * sizeof(double));
    for (int sid = 0; sid < nstates; ++sid) {
      float* ref = sid == 0 ? x : (sid <= N ? u[sid - 1] : v);
      oracle_state_stats(ref, 0, NULL, K, P, want);
      oracle_replica_mean(ref, 0, K, P);
      const double* got = hs + (size_t)sid * MTDAO_STATS_STRIDE;
      double big = 0.0;
      for (int k = 0; k < 4 + 2 * K; ++k) big = fmax(big, fabs(want[k]));
      for (int k = 0; k < 3 + 2 * K; ++k) {
        const int wi = k < 3 ? k : k + 1; /* oracle: [mean_sq, var, outer_sq, 0, sq[K], dot[K]] */
        const int gi = k < 3 ? k : (k < 3 + K ? MTDAO_STAT_WORKER_SQ + (k - 3) : MTDAO_STAT_WORKER_DOT + (k - 3 - K));
        const double den = fmax(fabs(want[wi]), 1e-6 * big);
        const double e = den > 0.0 ? fabs(got[gi] - want[wi]) / den : fabs(got[gi] - want[wi]);
        if (!(e <= stats_worst)) stats_worst = e;
      }
    }
    free(want);
    CHECK_HIP(hipFree(scratch));
  }

  /* every state of every worker, read back through the ABI */
  double worst = 0.0;
  for (int sid = 0; sid < nstates; ++sid) {
    const float* ref = sid == 0 ? x : (sid <= N ? u[sid - 1] : v);
    for (int32_t m = 0; m < K; ++m)
      CHECK_MT(h, mtdao_read_state(h, sid, m, 0, P, back + (int64_t)m * P, (void*)st));
    const double e = compare(back, ref, KP);
    if (!(e <= worst)) worst = e;
  }
  const int64_t count = mtdao_step_count(h);
  int64_t want_count = t->steps;
  if (W > 0) {
    /* the handle's host count moved during the capture only; the device count with every replay */
    mtdao_device_step ds;
    CHECK_HIP(hipMemcpy(&ds, dstep, sizeof ds, hipMemcpyDeviceToHost));
    if (ds.s != t->steps) {
      fprintf(stderr, "%s: device step count %lld, want %d\n", t->name, (long long)ds.s, t->steps);
      masks_ok = 0;
    }
    want_count = W;
    CHECK_HIP(hipGraphExecDestroy(gexec));
    CHECK_HIP(hipGraphDestroy(graph));
    CHECK_HIP(hipFree(dstep));
    CHECK_HIP(hipFree(dlr));
  }
  mtdao_destroy(h);
  const int ok = masks_ok && worst <= 1e-5 && stats_worst <= 1e-5 && count == want_count;
  printf("%s: K=%d P=%lld N=%d steps=%d state-syncs=%u max rel err %.3e", t->name, K, (long long)P, N, t->steps,
         nsync, worst);
  if (t->stats) printf(" diagnostics err %.3e", stats_worst);
  printf(" masks %s -> %s\n", masks_ok ? "match" : "DIFFER", ok ? "ok" : "FAIL");
  fflush(stdout);

  CHECK_HIP(hipFree(dx));
  for (int j = 0; j < N; ++j) CHECK_HIP(hipFree(du[j]));
  if (dv) CHECK_HIP(hipFree(dv));
  CHECK_HIP(hipFree(dg));
  if (ws) CHECK_HIP(hipFree(ws));
  CHECK_HIP(hipStreamDestroy(st));
  free(x);
  for (int j = 0; j < N; ++j) free(u[j]);
  free(v);
  free(g);
  free(back);
  return ok;
}

int main(void) {
  const drv_case cases[4] = {
      {"adam_n3_k4_step_sync", MTDAO_ADAM, 4, 3, 10007, {0.9f, 0.99f, 0.999f}, {0.3f, 0.3f, 0.3f}, 0.999f, 1e-8f,
       0.0f, 1e-3f, 4, {8, 8, 16}, 16, 32, 1, 0, 0},
      {"sgdm_n2_k5_clip_sync", MTDAO_SGDM, 5, 2, 8204, {0.9f, 0.99f}, {0.3f, 0.6f}, 0.0f, 0.0f, 0.05f, 1e-2f, 4,
       {2, 8}, 0, 24, 0, 0, 0},
      {"adam_n2_k6_sync_stats", MTDAO_ADAM, 6, 2, 4099, {0.9f, 0.99f}, {0.4f, 0.4f}, 0.999f, 1e-8f, 0.0f, 1e-3f, 4,
       {0, 0}, 0, 6, 0, 1, 0},
      {"adam_n2_k3_graph_device_step", MTDAO_ADAM, 3, 2, 4100, {0.9f, 0.99f}, {0.3f, 0.5f}, 0.999f, 1e-8f, 0.0f,
       1e-3f, 4, {8, 8}, 8, 24, 1, 0, 8},
  };
  int all = 1;
  for (int i = 0; i < 4; ++i) all &= run_case(&cases[i]);
  return all ? 0 : 1;
}
