/*
 * CPU oracle for the MT-DAO optimizer hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test-suite, the smoke check and the
 * benchmark's CPU-baseline leg may load this library.  It shares no code
 * with the GPU library and must never be used as a fallback for it.
 *
 * What it computes (paper: "Multi-timescale Distributed Adaptive Optimizers
 * with Local Updates", Section 2.3 Algorithm 1 = Adam form, Appendix
 * Algorithm 2 = ADOPT form, Appendix Algorithm 3 = SGDM form):
 *   one local step of every worker m for every element i, followed, at
 *   the caller's request, by the replica mean E_m[.] of one state; also
 *   the step of the probabilistic SGDM variant (Algorithm 4), the Nesterov
 *   OuterOpt at an averaging event of x, and the averaging diagnostics of
 *   one state (Section 4.1's metrics).
 * Arithmetic is IEEE double throughout.  Each state store rounds once to
 * its storage type (fp32 and bf16 with round-to-nearest-even, or fp64),
 * which puts the rounding points where a device kernel stores them.
 * Hyper-parameters arrive as the same fp32 values the GPU library gets and
 * are widened to double.  Plain scalar loops; no blocking, no fusion
 * beyond the order the algorithms give.
 *
 * Readings of the paper where it is silent or ambiguous (each is listed in
 * the design notes with its reason):
 *  - sync phase: after local update s (1-based), state S is averaged iff
 *    its period H_S > 0 and s mod H_S == 0 (Algorithm 1's schedule);
 *  - Adam bias correction, which Algorithm 1's caption omits: u_j / (1 -
 *    beta_j^s) and v / (1 - beta2^s) with the global step s, gradient term
 *    uncorrected; ADOPT and SGDM carry none;
 *  - Adam squares the clipped gradient in v;
 *  - clip(g, rho) is the per-worker global L2 norm clip, scale
 *    min(1, rho / ||g||), scale 1 for a zero norm;
 *  - ADOPT normalises by the second moment from before this step (the
 *    published ADOPT order: step 1 only sets v = g^2); the literal order of
 *    Algorithm 2 (normalise by the freshly updated v) is the "current"
 *    variant; clip(., c_t) is an element-wise clamp to [-c_t, c_t];
 *  - OuterOpt is the plain arithmetic mean unless the Nesterov OuterOpt is
 *    asked for (its reading is given where it is defined below).
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

#define OR_MAX_N 4

enum { OR_F32 = 0, OR_BF16 = 1, OR_F64 = 2 };
enum { OR_ADAM = 0, OR_ADOPT = 1, OR_SGDM = 2 };
enum { OR_ADOPT_PREV = 0, OR_ADOPT_CUR = 1 };

typedef struct {
  int32_t form;            /* OR_ADAM / OR_ADOPT / OR_SGDM                     */
  int32_t n;               /* number of first moments N, 1..4                  */
  int32_t x_dtype;         /* storage of x                                      */
  int32_t g_dtype;         /* storage of the gradient                           */
  int32_t m_dtype;         /* storage of u^j and v                              */
  int32_t bias_correction; /* Adam only: 1 = correct u^j and v                  */
  int32_t adopt_order;     /* OR_ADOPT_PREV / OR_ADOPT_CUR                      */
  float beta1[OR_MAX_N];   /* beta_{1,j}                                        */
  float omega[OR_MAX_N];   /* omega_j                                           */
  float beta2;             /* beta_2                                            */
  float eps;               /* epsilon                                           */
} oracle_cfg;

/* ---------------------------------------------------------------- storage */

/* Round a double to the nearest bf16 value (8 significant bits, fp32
 * exponent range, subnormal quantum 2^-133), ties to even; result is a
 * double holding that value exactly.  nearbyint() rounds ties to even in
 * the default floating-point environment. */
static double round_to_bf16(double a) {
  if (a == 0.0 || !isfinite(a)) return a;
  int e;
  frexp(a, &e);            /* |a| in [2^(e-1), 2^e) */
  int q = e - 8;           /* quantum for 8 significant bits */
  if (q < -133) q = -133;
  double r = ldexp(nearbyint(ldexp(a, -q)), q);
  const double bf16_max = ldexp(255.0, 120);
  if (fabs(r) > bf16_max) return copysign(INFINITY, a);
  return r;
}

static double load(const void* p, int32_t dt, int64_t i) {
  if (dt == OR_F32) return (double)((const float*)p)[i];
  if (dt == OR_BF16) {
    uint32_t b = (uint32_t)((const uint16_t*)p)[i] << 16;
    float f;
    memcpy(&f, &b, sizeof f);
    return (double)f;
  }
  return ((const double*)p)[i];
}

/* Store with one rounding to the storage type; returns the stored value. */
static double store(void* p, int32_t dt, int64_t i, double a) {
  if (dt == OR_F32) {
    float f = (float)a;
    ((float*)p)[i] = f;
    return (double)f;
  }
  if (dt == OR_BF16) {
    if (isnan(a)) {
      ((uint16_t*)p)[i] = 0x7FC0;
      return a;
    }
    float f = (float)round_to_bf16(a); /* exact: bf16 values are fp32 values */
    uint32_t b;
    memcpy(&b, &f, sizeof b);
    ((uint16_t*)p)[i] = (uint16_t)(b >> 16);
    return (double)f;
  }
  ((double*)p)[i] = a;
  return a;
}

static int64_t dtype_size(int32_t dt) { return dt == OR_F32 ? 4 : dt == OR_BF16 ? 2 : 8; }

/* ------------------------------------------------------------- schedule */

/* Which states are averaged after local update s (reading of the
 * "t mod K" conditions of Algorithms 1-3): bit 0 = x, bit j = u^j
 * (j = 1..N), bit N+1 = v (forms with a second moment only).  A period of
 * 0 means "never". */
uint32_t oracle_schedule(int64_t s, int32_t n, int32_t period_x, const int32_t* period_u,
                         int32_t period_v, int32_t has_v) {
  uint32_t mask = 0;
  if (period_x > 0 && s % period_x == 0) mask |= 1u;
  for (int32_t j = 0; j < n; ++j)
    if (period_u[j] > 0 && s % period_u[j] == 0) mask |= 1u << (j + 1);
  if (has_v && period_v > 0 && s % period_v == 0) mask |= 1u << (n + 1);
  return mask;
}

/* ------------------------------------------------------ clip(g, rho) */

/* Sum of squares of n stored gradient values, in double (the square of the
 * L2 norm in clip(g, rho), Algorithm 1 and Algorithm 3). */
double oracle_sumsq(const void* g, int32_t g_dtype, int64_t n) {
  double acc = 0.0;
  for (int64_t i = 0; i < n; ++i) {
    double a = load(g, g_dtype, i);
    acc += a * a;
  }
  return acc;
}

/* Scale factor of the global-norm clip: min(1, rho / norm); 1 when the clip
 * is off (rho <= 0) or the norm is zero. */
double oracle_clip_scale(double norm, double rho) {
  if (!(rho > 0.0) || norm == 0.0) return 1.0;
  double c = rho / norm;
  return c < 1.0 ? c : 1.0;
}

/* ------------------------------------------------------------ local step */

/*
 * One local update of every worker (rows m = 0..K-1, row stride P).
 *   s      global 1-based step number of this update
 *   lr     eta_t for this update
 *   clip_c ADOPT c_t (<= 0: no clamp); ignored by Adam and SGDM
 *   scale  per-worker clip factor from oracle_clip_scale (NULL: all 1)
 * The base values x_bar, u_bar, v_bar are whatever the buffers hold (after
 * the previous step's averaging, if any).
 */
void oracle_local_step(const oracle_cfg* c, int64_t s, float lr, float clip_c, const double* scale,
                       void* x, void* const* u, void* v, const void* g, int64_t K, int64_t P) {
  const int32_t n = c->n;
  double beta[OR_MAX_N], omega[OR_MAX_N], bc[OR_MAX_N];
  double omega_sum = 0.0;
  for (int32_t j = 0; j < n; ++j) {
    beta[j] = (double)c->beta1[j];
    omega[j] = (double)c->omega[j];
    omega_sum += omega[j];
    bc[j] = 1.0;
  }
  const double g_weight = 1.0 - omega_sum;   /* weight of the current gradient */
  const double beta2 = (double)c->beta2;
  const double eps = (double)c->eps;
  const double eta = (double)lr;
  double bc2 = 1.0;
  if (c->form == OR_ADAM && c->bias_correction) {
    for (int32_t j = 0; j < n; ++j) bc[j] = 1.0 - pow(beta[j], (double)s);
    bc2 = 1.0 - pow(beta2, (double)s);
  }
  const double cc = (double)clip_c;

  for (int64_t m = 0; m < K; ++m) {
    const double sm = scale ? scale[m] : 1.0;
    for (int64_t p = 0; p < P; ++p) {
      const int64_t i = m * P + p;
      const double graw = load(g, c->g_dtype, i);

      if (c->form == OR_ADAM) {
        /* Algorithm 1: clipped gradient, N EMAs, second moment, QH step. */
        const double gh = sm * graw;
        double num = g_weight * gh;
        for (int32_t j = 0; j < n; ++j) {
          double uj = beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gh;
          uj = store(u[j], c->m_dtype, i, uj);
          num += omega[j] * (uj / bc[j]);
        }
        double vv = beta2 * load(v, c->m_dtype, i) + (1.0 - beta2) * gh * gh;
        vv = store(v, c->m_dtype, i, vv);
        const double delta = num / (sqrt(vv / bc2) + eps);
        store(x, c->x_dtype, i, load(x, c->x_dtype, i) - eta * delta);
      } else if (c->form == OR_ADOPT) {
        /* Algorithm 2: normalise by the second moment, clamp, N EMAs of the
         * clamped normalised gradient, QH combination without further
         * normalisation. */
        double vv = load(v, c->m_dtype, i);
        double gn;
        if (c->adopt_order == OR_ADOPT_PREV) {
          if (s == 1) { /* the first gradient only initialises v */
            store(v, c->m_dtype, i, graw * graw);
            continue;
          }
          gn = graw / (sqrt(vv) + eps);
          vv = beta2 * vv + (1.0 - beta2) * graw * graw;
          store(v, c->m_dtype, i, vv);
        } else {
          vv = beta2 * vv + (1.0 - beta2) * graw * graw;
          vv = store(v, c->m_dtype, i, vv);
          gn = graw / (sqrt(vv) + eps);
        }
        if (cc > 0.0) gn = gn > cc ? cc : (gn < -cc ? -cc : gn);
        double delta = g_weight * gn;
        for (int32_t j = 0; j < n; ++j) {
          double uj = beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gn;
          uj = store(u[j], c->m_dtype, i, uj);
          delta += omega[j] * uj;
        }
        store(x, c->x_dtype, i, load(x, c->x_dtype, i) - eta * delta);
      } else {
        /* Algorithm 3: clipped gradient, N EMAs, unnormalised QH step. */
        const double gh = sm * graw;
        double delta = g_weight * gh;
        for (int32_t j = 0; j < n; ++j) {
          double uj = beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gh;
          uj = store(u[j], c->m_dtype, i, uj);
          delta += omega[j] * uj;
        }
        store(x, c->x_dtype, i, load(x, c->x_dtype, i) - eta * delta);
      }
    }
  }
}

/* ------------------------------------------- probabilistic variant */

/*
 * One step of the probabilistic SGDM variant (Algorithm 4) given this
 * step's averaging events in mask (bit 0 = x, bit j = u^j), which the
 * caller draws: for every element, each first moment of every worker is
 * updated and, when its event fires, replaced by its worker mean BEFORE the
 * update direction uses it; x of every worker is updated with that
 * direction and, when its event fires, replaced by its worker mean.
 * The gradient term (1 - sum omega) is kept for generality (Algorithm 4
 * has sum omega = 1, so it is zero there); scale as in oracle_local_step.
 */
void oracle_sgdm_prob_step(const oracle_cfg* c, float lr, uint32_t mask, const double* scale, void* x,
                           void* const* u, const void* g, int64_t K, int64_t P) {
  const int32_t n = c->n;
  double beta[OR_MAX_N], omega[OR_MAX_N], omega_sum = 0.0;
  for (int32_t j = 0; j < n; ++j) {
    beta[j] = (double)c->beta1[j];
    omega[j] = (double)c->omega[j];
    omega_sum += omega[j];
  }
  const double g_weight = 1.0 - omega_sum;
  const double eta = (double)lr;
  for (int64_t p = 0; p < P; ++p) {
    for (int32_t j = 0; j < n; ++j) {
      for (int64_t m = 0; m < K; ++m) {
        const int64_t i = m * P + p;
        const double gh = (scale ? scale[m] : 1.0) * load(g, c->g_dtype, i);
        store(u[j], c->m_dtype, i, beta[j] * load(u[j], c->m_dtype, i) + (1.0 - beta[j]) * gh);
      }
      if (mask & (1u << (j + 1))) {
        double acc = 0.0;
        for (int64_t m = 0; m < K; ++m) acc += load(u[j], c->m_dtype, m * P + p);
        for (int64_t m = 0; m < K; ++m) store(u[j], c->m_dtype, m * P + p, acc / (double)K);
      }
    }
    for (int64_t m = 0; m < K; ++m) {
      const int64_t i = m * P + p;
      const double gh = (scale ? scale[m] : 1.0) * load(g, c->g_dtype, i);
      double delta = g_weight * gh;
      for (int32_t j = 0; j < n; ++j) delta += omega[j] * load(u[j], c->m_dtype, i);
      store(x, c->x_dtype, i, load(x, c->x_dtype, i) - eta * delta);
    }
    if (mask & 1u) {
      double acc = 0.0;
      for (int64_t m = 0; m < K; ++m) acc += load(x, c->x_dtype, m * P + p);
      for (int64_t m = 0; m < K; ++m) store(x, c->x_dtype, m * P + p, acc / (double)K);
    }
  }
}

/* --------------------------------------------------------- replica mean */

/* E_m[S]: the arithmetic mean over the K workers of one state, written back
 * to every worker's row (Algorithms 1-3, OuterOpt = averaging). */
void oracle_replica_mean(void* state, int32_t dtype, int64_t K, int64_t P) {
  for (int64_t p = 0; p < P; ++p) {
    double acc = 0.0;
    for (int64_t m = 0; m < K; ++m) acc += load(state, dtype, m * P + p);
    const double mean = acc / (double)K;
    for (int64_t m = 0; m < K; ++m) store(state, dtype, m * P + p, mean);
  }
}

/* -------------------------------------------------- Nesterov OuterOpt */

/*
 * OuterOpt = Nesterov momentum at an averaging event of x (the outer
 * optimizer the paper compares against; the outer Nesterov step of the
 * local-update literature): with the workers' mean xbar = E_m[x^m], the
 * outer parameters xo and the outer momentum b (fp32 [P] each),
 *   d  = xo - xbar            (outer pseudo-gradient)
 *   b  = mu * b + d
 *   xo = xo - outer_lr * (d + mu * b)
 * and every worker restarts from xo.  outer_lr = 1, mu = 0 gives xo = xbar,
 * plain averaging.
 */
void oracle_outer_nesterov(void* x, int32_t x_dtype, float* xo, float* b, float outer_lr, float mu, int64_t K,
                           int64_t P) {
  const double lr = (double)outer_lr, m_ = (double)mu;
  for (int64_t p = 0; p < P; ++p) {
    double acc = 0.0;
    for (int64_t m = 0; m < K; ++m) acc += load(x, x_dtype, m * P + p);
    const double xbar = acc / (double)K;
    const double d = (double)xo[p] - xbar;
    const double bn = m_ * (double)b[p] + d;
    b[p] = (float)bn;
    const double xn = (double)xo[p] - lr * (d + m_ * (double)b[p]);
    xo[p] = (float)xn;
    for (int64_t m = 0; m < K; ++m) store(x, x_dtype, m * P + p, (double)xo[p]);
  }
}

/* ------------------------------------------------ averaging diagnostics */

/*
 * Diagnostics of one state across the workers (Section 4.1, other
 * metrics: cross-worker variance, relative change, cosine alignment), from
 * the values before they are averaged.  With xo == NULL the vectors are the
 * workers' states c^m = S^m; with the outer parameters xo of a Nesterov
 * OuterOpt they are the workers' pseudo-gradients c^m = xo - x^m.  cbar is
 * their mean.  out (4 + 2 K doubles):
 *   out[0] = ||cbar||^2
 *   out[1] = (1/K) sum_m ||c^m - cbar||^2      (cross-worker variance)
 *   out[2] = ||xo||^2 (0 without xo)           (relative change = sqrt(out[0] / out[2]))
 *   out[3] = 0
 *   out[4 + m]     = ||c^m||^2
 *   out[4 + K + m] = <c^m, cbar>               (cosine = out[4+K+m] / sqrt(out[4+m] out[0]))
 */
void oracle_state_stats(const void* s, int32_t dtype, const float* xo, int64_t K, int64_t P, double* out) {
  for (int64_t k = 0; k < 4 + 2 * K; ++k) out[k] = 0.0;
  for (int64_t p = 0; p < P; ++p) {
    double cbar = 0.0;
    for (int64_t m = 0; m < K; ++m) {
      const double v = load(s, dtype, m * P + p);
      cbar += xo ? (double)xo[p] - v : v;
    }
    cbar /= (double)K;
    out[0] += cbar * cbar;
    if (xo) out[2] += (double)xo[p] * (double)xo[p];
    for (int64_t m = 0; m < K; ++m) {
      const double v = load(s, dtype, m * P + p);
      const double c = xo ? (double)xo[p] - v : v;
      out[1] += (c - cbar) * (c - cbar);
      out[4 + m] += c * c;
      out[4 + K + m] += c * cbar;
    }
  }
  out[1] /= (double)K;
}

/* Size in bytes of one element of a storage type (for the Python side). */
int64_t oracle_dtype_size(int32_t dtype) { return dtype_size(dtype); }
