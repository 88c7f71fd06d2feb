// Host side of the MT-DAO C ABI (include/mtdao.h): validation, the sync
// schedule, per-step scalars, launch configuration and error mapping.
// The arithmetic of every step runs in the kernels of kernels.hpp.

#include <hip/hip_runtime.h>
#include <rocprofiler-sdk-roctx/roctx.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstddef>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <type_traits>
#include <vector>

#include "../../include/mtdao.h"
#include "kernels.hpp"

using namespace mtdao;

static_assert(sizeof(DeviceStep) == sizeof(mtdao_device_step) && offsetof(DeviceStep, s) == offsetof(mtdao_device_step, s),
              "DeviceStep mirrors mtdao_device_step");

struct mtdao_handle {
  mtdao_config cfg;                 // copy; tensor_numel points into `tensors`
  std::vector<int64_t> tensors;
  void* x = nullptr;
  float* u[MTDAO_MAX_N] = {nullptr, nullptr, nullptr, nullptr};
  float* v = nullptr;
  float* x_outer = nullptr;         // Nesterov OuterOpt: outer parameters [P]
  float* x_outer_mom = nullptr;     // Nesterov OuterOpt: outer momentum [P]
  float* scale = nullptr;           // workspace: [K] clip factors
  double* partials = nullptr;       // workspace: [K][norm_blocks]
  int32_t norm_blocks = 0;
  int64_t s = 0;                    // local updates applied
  int64_t outer_done_s = -1;        // Nesterov: step s whose outer step has run
  int64_t dev_base = 0;             // host count at the last device-step set or advance
  std::string err;
};

namespace {

thread_local std::string g_err;

// roctx ranges around every enqueueing call, for timelines of
// rocprofv3 --marker-trace: on when MTDAO_ROCTX=1 in the environment.
bool roctx_on() {
  static const bool on = [] {
    const char* e = std::getenv("MTDAO_ROCTX");
    return e != nullptr && e[0] == '1';
  }();
  return on;
}

struct RoctxRange {
  bool on;
  explicit RoctxRange(const char* fmt, ...) : on(roctx_on()) {
    if (!on) return;
    char buf[128];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    roctxRangePushA(buf);
  }
  ~RoctxRange() {
    if (on) roctxRangePop();
  }
};

// Vector slots per thread in the local step: one for every form (measured
// on MI355X with 1 KiB pieces: two slots were 0-0.5 % slower for Adam's
// 6-read/5-write stream and equal for SGDM and ADOPT).
constexpr int step_slots(int) { return 1; }
// Piece length of the tile -> element map (tile_elem): one wavefront's
// access, 64 lanes of V elements (1 KiB of fp32 for V = 4).
constexpr int piece_for(int V) { return 64 * V; }
constexpr int kStepNT = 3;     // nontemporal hints of the local step (bit 0 loads, bit 1 stores)
constexpr bool kMeanNT = true; // nontemporal hints of the replica mean
constexpr int kNormU = 8;      // vector slots per thread in the norm pass

int32_t fail(std::string* sink, int32_t code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  *sink = buf;
  return code;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }
int64_t esize(int32_t dt) { return dt == MTDAO_BF16 ? 2 : 4; }
bool has_v(const mtdao_config& c) { return c.form != MTDAO_SGDM; }

// Vector width of a row: 16-byte slots when every row start stays aligned.
int vec_width(int32_t dtype_small, int64_t P) {
  const int v = dtype_small == MTDAO_BF16 ? 8 : 4;
  return (P % v == 0) ? v : 1;
}

int32_t validate(const mtdao_config* c, std::string* e) {
  if (!c) return fail(e, MTDAO_ERR_INVALID_ARG, "config is NULL");
  if (c->form < MTDAO_ADAM || c->form > MTDAO_SGDM)
    return fail(e, MTDAO_ERR_INVALID_ARG, "form %d is not ADAM(0), ADOPT(1) or SGDM(2)", c->form);
  if (c->replicas < 1 || c->replicas > MTDAO_MAX_REPLICAS)
    return fail(e, MTDAO_ERR_INVALID_ARG, "replicas %d outside [1, %d]", c->replicas, MTDAO_MAX_REPLICAS);
  if (c->n_moments < 1 || c->n_moments > MTDAO_MAX_N)
    return fail(e, MTDAO_ERR_INVALID_ARG, "n_moments %d outside [1, %d]", c->n_moments, MTDAO_MAX_N);
  if ((c->param_dtype != MTDAO_F32 && c->param_dtype != MTDAO_BF16) ||
      (c->grad_dtype != MTDAO_F32 && c->grad_dtype != MTDAO_BF16))
    return fail(e, MTDAO_ERR_INVALID_ARG, "param_dtype/grad_dtype must be F32(0) or BF16(1)");
  if (c->adopt_order != MTDAO_ADOPT_PREV && c->adopt_order != MTDAO_ADOPT_CUR)
    return fail(e, MTDAO_ERR_INVALID_ARG, "adopt_order %d is not PREV(0) or CUR(1)", c->adopt_order);
  if (c->bias_correction != 0 && c->bias_correction != 1)
    return fail(e, MTDAO_ERR_INVALID_ARG, "bias_correction must be 0 or 1");
  double wsum = 0.0;
  for (int j = 0; j < c->n_moments; ++j) {
    const float b = c->beta1[j], w = c->omega[j];
    if (!(b >= 0.0f && b < 1.0f)) return fail(e, MTDAO_ERR_INVALID_ARG, "beta1[%d]=%g outside [0,1)", j, b);
    if (!(w >= 0.0f && w <= 1.0f)) return fail(e, MTDAO_ERR_INVALID_ARG, "omega[%d]=%g outside [0,1]", j, w);
    if (c->period_u[j] < 0) return fail(e, MTDAO_ERR_INVALID_ARG, "period_u[%d]=%d < 0", j, c->period_u[j]);
    wsum += (double)w;
  }
  if (wsum > 1.0 + 1e-6) return fail(e, MTDAO_ERR_INVALID_ARG, "sum of omega = %.9g exceeds 1", wsum);
  if (has_v(*c)) {
    if (!(c->beta2 >= 0.0f && c->beta2 < 1.0f))
      return fail(e, MTDAO_ERR_INVALID_ARG, "beta2=%g outside [0,1)", c->beta2);
    if (!(c->eps >= 0.0f) || !std::isfinite(c->eps))
      return fail(e, MTDAO_ERR_INVALID_ARG, "eps=%g must be finite and >= 0", c->eps);
    if (c->period_v < 0) return fail(e, MTDAO_ERR_INVALID_ARG, "period_v=%d < 0", c->period_v);
  }
  if (!std::isfinite(c->clip_rho)) return fail(e, MTDAO_ERR_INVALID_ARG, "clip_rho is not finite");
  if (c->form == MTDAO_ADOPT && c->clip_rho > 0.0f)
    return fail(e, MTDAO_ERR_INVALID_ARG, "ADOPT clips the normalised gradient with c_t (per call), not rho");
  if (c->period_x < 0) return fail(e, MTDAO_ERR_INVALID_ARG, "period_x=%d < 0", c->period_x);
  if (c->sync_order != MTDAO_SYNC_AFTER_STEP && c->sync_order != MTDAO_SYNC_MOMENTA_IN_STEP)
    return fail(e, MTDAO_ERR_INVALID_ARG, "sync_order %d is not AFTER_STEP(0) or MOMENTA_IN_STEP(1)", c->sync_order);
  if (c->sync_order == MTDAO_SYNC_MOMENTA_IN_STEP && c->form != MTDAO_SGDM)
    return fail(e, MTDAO_ERR_INVALID_ARG, "sync_order MOMENTA_IN_STEP is the SGDM variant (Algorithm 4)");
  if (c->outer_opt != MTDAO_OUTER_AVERAGE && c->outer_opt != MTDAO_OUTER_NESTEROV)
    return fail(e, MTDAO_ERR_INVALID_ARG, "outer_opt %d is not AVERAGE(0) or NESTEROV(1)", c->outer_opt);
  if (c->outer_opt == MTDAO_OUTER_NESTEROV) {
    if (!(c->outer_lr > 0.0f) || !std::isfinite(c->outer_lr))
      return fail(e, MTDAO_ERR_INVALID_ARG, "outer_lr=%g must be finite and > 0", c->outer_lr);
    if (!(c->outer_momentum >= 0.0f && c->outer_momentum < 1.0f))
      return fail(e, MTDAO_ERR_INVALID_ARG, "outer_momentum=%g outside [0,1)", c->outer_momentum);
    if (c->sync_order != MTDAO_SYNC_AFTER_STEP)
      return fail(e, MTDAO_ERR_INVALID_ARG, "the Nesterov OuterOpt needs sync_order AFTER_STEP");
  }
  if (c->start_step < 0) return fail(e, MTDAO_ERR_INVALID_ARG, "start_step < 0");
  if (c->numel < 0) return fail(e, MTDAO_ERR_INVALID_ARG, "numel < 0");
  if (c->numel > (INT64_C(1) << 40) / c->replicas)
    return fail(e, MTDAO_ERR_INVALID_ARG, "replicas * numel exceeds 2^40 elements");
  if (c->n_tensors < 0) return fail(e, MTDAO_ERR_INVALID_ARG, "n_tensors < 0");
  if (c->n_tensors > 0) {
    if (!c->tensor_numel) return fail(e, MTDAO_ERR_INVALID_ARG, "tensor_numel is NULL");
    int64_t sum = 0;
    for (int32_t t = 0; t < c->n_tensors; ++t) {
      if (c->tensor_numel[t] < 0) return fail(e, MTDAO_ERR_INVALID_ARG, "tensor_numel[%d] < 0", t);
      sum += c->tensor_numel[t];
      if (sum > c->numel) break;
    }
    if (sum != c->numel)
      return fail(e, MTDAO_ERR_INVALID_ARG, "tensor_numel does not sum to numel=%lld", (long long)c->numel);
  }
  return MTDAO_OK;
}

uint32_t schedule_mask(const mtdao_config& c, int64_t s) {
  uint32_t mask = 0;
  if (c.period_x > 0 && s % c.period_x == 0) mask |= 1u;
  for (int j = 0; j < c.n_moments; ++j)
    if (c.period_u[j] > 0 && s % c.period_u[j] == 0) mask |= 1u << (j + 1);
  if (has_v(c) && c.period_v > 0 && s % c.period_v == 0) mask |= 1u << (c.n_moments + 1);
  return mask;
}

uint32_t valid_bits(const mtdao_config& c) {
  const int nb = 1 + c.n_moments + (has_v(c) ? 1 : 0);
  return (nb >= 32) ? 0xFFFFFFFFu : ((1u << nb) - 1u);
}

// Workgroups per replica of the norm pass: one tile of kBlock * V * kNormU
// elements each, so the grid (tiles, K) is dispatched replica by replica
// and the pass streams one row at a time, like a plain read.  (A fixed
// grid of a few hundred looping workgroups per replica keeps every row in
// flight at once: 16 concurrent read streams at K = 16.)  One fp64 partial
// per workgroup; P <= 2^40 keeps the count below 2^31.
int32_t norm_blocks_for(int64_t P) {
  const int V = (P % 4 == 0) ? 4 : 1;
  const int64_t nb = V == 4 ? tiles_for<kBlock * 4 * kNormU, piece_for(4)>(P)
                            : tiles_for<kBlock * kNormU, piece_for(1)>(P);
  return (int32_t)(nb < 1 ? 1 : nb);
}

size_t workspace_for(const mtdao_config& c) {
  if (!(c.clip_rho > 0.0f) || c.form == MTDAO_ADOPT) return 0;
  const size_t scale_bytes = ((size_t)c.replicas * sizeof(float) + 255) / 256 * 256;
  return scale_bytes + (size_t)c.replicas * (size_t)norm_blocks_for(c.numel) * sizeof(double);
}

// Non-overlap of two [lo, lo + bytes) device ranges.
bool overlap(const void* a, int64_t abytes, const void* b, int64_t bbytes) {
  const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
  return a0 < b0 + (uintptr_t)bbytes && b0 < a0 + (uintptr_t)abytes;
}

int32_t hip_check(std::string* e, hipError_t r, const char* what) {
  if (r != hipSuccess) return fail(e, MTDAO_ERR_HIP, "%s: %s", what, hipGetErrorString(r));
  return MTDAO_OK;
}

dim3 grid_for(int64_t tiles, int32_t ny) {
  const int64_t maxx = INT64_C(0x7fffffff);
  return dim3((unsigned)(tiles < maxx ? (tiles > 0 ? tiles : 1) : maxx), (unsigned)ny, 1);
}

// ---------------------------------------------------------------- dispatch

template <int V>
using IntC = std::integral_constant<int, V>;
template <typename T>
struct TypeC {
  using type = T;
};

// Calls f(form, n, xtype, gtype, vwidth) with compile-time constants for the
// configuration of c and the runtime vector width V (4, or 1 when a row
// length breaks the 4-element alignment of row starts).
template <typename F>
void dispatch_step(const mtdao_config& c, int V, F&& f) {
  auto with_types = [&](auto form, auto n) {
    auto with_v = [&](auto xt, auto gt) {
      // 4-element slots: 16-byte fp32 and 8-byte bf16 accesses per lane
      if (V == 1) f(form, n, xt, gt, IntC<1>{});
      else f(form, n, xt, gt, IntC<4>{});
    };
    if (c.param_dtype == MTDAO_F32 && c.grad_dtype == MTDAO_F32) with_v(TypeC<float>{}, TypeC<float>{});
    else if (c.param_dtype == MTDAO_F32) with_v(TypeC<float>{}, TypeC<uint16_t>{});
    else if (c.grad_dtype == MTDAO_F32) with_v(TypeC<uint16_t>{}, TypeC<float>{});
    else with_v(TypeC<uint16_t>{}, TypeC<uint16_t>{});
  };
  auto with_form = [&](auto form) {
    switch (c.n_moments) {
      case 1: with_types(form, IntC<1>{}); break;
      case 2: with_types(form, IntC<2>{}); break;
      case 3: with_types(form, IntC<3>{}); break;
      default: with_types(form, IntC<4>{}); break;
    }
  };
  if (c.form == MTDAO_ADAM) with_form(IntC<kAdam>{});
  else if (c.form == MTDAO_ADOPT) with_form(IntC<kAdopt>{});
  else with_form(IntC<kSgdm>{});
}

// The local step alone: grid (tiles of one row, K).
void launch_step(const mtdao_config& c, StepParams p, int V, hipStream_t st) {
  dispatch_step(c, V, [&](auto form, auto n, auto xt, auto gt, auto vw) {
    constexpr int FORM = decltype(form)::value, N = decltype(n)::value, VV = decltype(vw)::value;
    using XT = typename decltype(xt)::type;
    using GT = typename decltype(gt)::type;
    constexpr int U = step_slots(FORM), C = piece_for(VV), T = kBlock * VV * U;
    // every stream read at two places at once: rows m and m + ceil(K/2)
    // when K > 1, else the two halves [0, wlen) and [wlen, P) of the row
    auto go = [&](auto win) {
      constexpr int WIN = decltype(win)::value;
      dim3 grid;
      if constexpr (WIN == kWinPairs) {
        p.tiles = 2 * tiles_for<T, C>(p.P);
        grid = grid_for(p.tiles, (c.replicas + 1) / 2);
      } else {
        p.wlen = ((p.P + 1) / 2 + T - 1) / T * T;
        if (p.wlen > p.P) p.wlen = p.P;
        p.tiles = 2 * tiles_for<T, C>(p.wlen);
        grid = grid_for(p.tiles, c.replicas);
      }
      if constexpr (FORM == kAdopt) {
        if (c.adopt_order == MTDAO_ADOPT_CUR) {
          hipLaunchKernelGGL((k_local_step<FORM, N, XT, GT, VV, U, kStepNT, kCur, kBlock, C, WIN>), grid, dim3(kBlock),
                             0, st, p);
          return;
        }
      }
      hipLaunchKernelGGL((k_local_step<FORM, N, XT, GT, VV, U, kStepNT, kPrev, kBlock, C, WIN>), grid, dim3(kBlock), 0,
                         st, p);
    };
    if (c.replicas > 1) go(IntC<kWinPairs>{});
    else go(IntC<kWinHalves>{});
  });
}

// The local step with the replica mean of the states in mask: grid over
// tiles of one row, each thread covering all K replicas of its columns.
void launch_step_sync(const mtdao_config& c, StepParams p, int V, uint32_t mask, hipStream_t st) {
  dispatch_step(c, V, [&](auto form, auto n, auto xt, auto gt, auto vw) {
    constexpr int FORM = decltype(form)::value, N = decltype(n)::value, VV = decltype(vw)::value;
    using XT = typename decltype(xt)::type;
    using GT = typename decltype(gt)::type;
    if (c.replicas > 1 && c.replicas <= kWaveMaxK) {
      // one wavefront per replica
      const int64_t per = (int64_t)64 * VV;
      p.tiles = (p.P + per - 1) / per;
      const dim3 grid = grid_for(p.tiles, 1), block(64 * c.replicas);
      if constexpr (FORM == kAdopt) {
        if (c.adopt_order == MTDAO_ADOPT_CUR) {
          hipLaunchKernelGGL((k_local_step_sync_waves<FORM, N, XT, GT, VV, kStepNT, kCur>), grid, block, 0, st, p, mask,
                             c.replicas);
          return;
        }
      }
      hipLaunchKernelGGL((k_local_step_sync_waves<FORM, N, XT, GT, VV, kStepNT, kPrev>), grid, block, 0, st, p, mask,
                         c.replicas);
      return;
    }
    constexpr int C = piece_for(VV);
    p.tiles = tiles_for<kBlock * VV, C>(p.P);
    const dim3 grid = grid_for(p.tiles, 1);
    if constexpr (FORM == kAdopt) {
      if (c.adopt_order == MTDAO_ADOPT_CUR) {
        hipLaunchKernelGGL((k_local_step_sync<FORM, N, XT, GT, VV, kStepNT, kCur, C>), grid, dim3(kBlock), 0, st, p,
                           mask, c.replicas);
        return;
      }
    }
    hipLaunchKernelGGL((k_local_step_sync<FORM, N, XT, GT, VV, kStepNT, kPrev, C>), grid, dim3(kBlock), 0, st, p,
                       mask, c.replicas);
  });
}

template <typename GT>
void launch_adopt_init(const void* g, float* v, int64_t P, int32_t K, int V, hipStream_t st) {
  const int64_t per = (int64_t)kBlock * 2;
  if (V == 1) {
    hipLaunchKernelGGL((k_adopt_init_v<GT, 1, 2, false>), grid_for((P + per - 1) / per, K), dim3(kBlock), 0, st,
                       g, v, P, (P + per - 1) / per);
  } else {
    hipLaunchKernelGGL((k_adopt_init_v<GT, 4, 2, false>), grid_for((P + 4 * per - 1) / (4 * per), K), dim3(kBlock),
                       0, st, g, v, P, (P + 4 * per - 1) / (4 * per));
  }
}

template <typename GT>
void launch_norm(const void* g, int64_t P, int32_t K, int V, int32_t nb, double* partials, hipStream_t st) {
  if (V == 1) {
    constexpr int C = piece_for(1);
    hipLaunchKernelGGL((k_sumsq_partial<GT, 1, kNormU, C>), dim3(nb, K), dim3(kBlock), 0, st, g, P,
                       tiles_for<kBlock * kNormU, C>(P), partials);
  } else {
    constexpr int C = piece_for(4);
    hipLaunchKernelGGL((k_sumsq_partial<GT, 4, kNormU, C>), dim3(nb, K), dim3(kBlock), 0, st, g, P,
                       tiles_for<kBlock * 4 * kNormU, C>(P), partials);
  }
}

template <typename T>
void launch_mean(MeanParams p, int nstates, int V, hipStream_t st) {
  constexpr int VW = sizeof(T) == 2 ? 8 : 4;  // elements of a 16-byte slot
  if (p.K > 1 && p.K <= kWaveMaxK) {
    // one piece of 64 V elements per workgroup; one wavefront per replica,
    // or per two replicas for even K > 8 and for bf16 rows at K = 8
    // (measured on MI355X at K = 8: bf16 x 72% of peak with two rows per
    // wave against 68% with one, fp32 states 75.7% against 77.2%)
    const int vw = V == 1 ? 1 : VW;
    p.tiles = (p.P + 64 * vw - 1) / (64 * vw);
    const bool two = p.K % 2 == 0 && (p.K > 8 || (p.K == 8 && sizeof(T) == 2));
    const dim3 grid = grid_for(p.tiles, nstates), block(64 * (two ? p.K / 2 : p.K));
    const size_t lds = (size_t)p.K * 64 * vw * sizeof(float);
    if (two) {
      if (vw == 1) hipLaunchKernelGGL((k_replica_mean_waves<T, 1, kMeanNT, 2>), grid, block, lds, st, p);
      else hipLaunchKernelGGL((k_replica_mean_waves<T, VW, kMeanNT, 2>), grid, block, lds, st, p);
    } else {
      if (vw == 1) hipLaunchKernelGGL((k_replica_mean_waves<T, 1, kMeanNT>), grid, block, lds, st, p);
      else hipLaunchKernelGGL((k_replica_mean_waves<T, VW, kMeanNT>), grid, block, lds, st, p);
    }
    return;
  }
  // K = 1 (an outer step only) and K > kWaveMaxK: one thread per column
  if (V == 1) {
    p.tiles = tiles_for<kBlock, piece_for(1)>(p.P);
    hipLaunchKernelGGL((k_replica_mean<T, 1, kMeanNT, 1, piece_for(1)>), grid_for(p.tiles, nstates), dim3(kBlock), 0,
                       st, p);
  } else {
    p.tiles = tiles_for<VW * kBlock, piece_for(VW)>(p.P);
    hipLaunchKernelGGL((k_replica_mean<T, VW, kMeanNT, 1, piece_for(VW)>), grid_for(p.tiles, nstates), dim3(kBlock),
                       0, st, p);
  }
}

// The diagnostics pass of nstates states of one storage type: V elements
// per lane (16-byte accesses, or 1 when a row length breaks alignment), K
// waves per workgroup, kStatsPieces pieces per workgroup, then the two
// fixed-order reduction levels into out.  partials holds
// nstates * kStatsSums(K) * (workgroups + chunks) doubles.
//
// Pieces per workgroup, measured on MI355X at 1.31B params x 4 replicas
// (one state, DPP wave sums): 2 -> 7.65 ms, 3 -> 7.3 ms, 4 -> 6.9 ms,
// 6 -> 7.35 ms, 8 -> 7.3 ms.  With shuffle-based wave sums the closing
// reduction of each workgroup dominated below 4 (1 -> 14.5 ms, 2 -> 9.5 ms).
constexpr int32_t kStatsPieces = 4;
int64_t stats_pieces(int64_t P, int V) { return (P + 64 * V - 1) / (64 * V); }
int64_t stats_blocks(int64_t pieces) { return (pieces + 8 * kStatsPieces - 1) / (8 * kStatsPieces) * 8; }
int64_t stats_chunks(int64_t nb) { return (nb + kStatsChunk - 1) / kStatsChunk; }

template <typename T>
void launch_stats(MeanParams q, int nstates, int V, double* partials, double* out, hipStream_t st) {
  q.tiles = stats_pieces(q.P, V);
  const dim3 grid((unsigned)stats_blocks(q.tiles), nstates), block(64 * q.K);
  const int64_t nb = grid.x, nc = stats_chunks(nb);
  const int32_t ns = kStatsSums(q.K);
  double* level1 = partials + (size_t)nstates * ns * nb;
  const size_t lds = (size_t)q.K * 64 * V * sizeof(float);
  constexpr int VV = sizeof(T) == 2 ? 8 : 4;
  if (V == 1) hipLaunchKernelGGL((k_replica_mean_stats<T, 1>), grid, block, lds, st, q, kStatsPieces, partials);
  else hipLaunchKernelGGL((k_replica_mean_stats<T, VV>), grid, block, lds, st, q, kStatsPieces, partials);
  hipLaunchKernelGGL(k_stats_reduce, dim3((unsigned)nc, nstates), dim3(256), 0, st, partials, nb, ns, level1);
  hipLaunchKernelGGL(k_stats_finalize, dim3(nstates), dim3(256), 0, st, level1, (int32_t)nc, q.K, out);
}

// Doubles of the diagnostics scratch for up to 2 + N fp32 states and a bf16
// x: each launch's partials and chunk sums, then the finalized rows of the
// two launches.
size_t stats_scratch_doubles(const mtdao_config& c, size_t* fp32_part, size_t* bf16_part) {
  const int64_t ns = kStatsSums(c.replicas);
  const int64_t nb32 = stats_blocks(stats_pieces(c.numel, vec_width(MTDAO_F32, c.numel)));
  const int64_t nb16 = stats_blocks(stats_pieces(c.numel, vec_width(MTDAO_BF16, c.numel)));
  *fp32_part = (size_t)(2 + c.n_moments) * ns * (nb32 + stats_chunks(nb32));
  *bf16_part = c.param_dtype == MTDAO_BF16 ? (size_t)ns * (nb16 + stats_chunks(nb16)) : 0;
  return *fp32_part + *bf16_part + (size_t)2 * (2 + kMaxN) * kStatsStride;
}

size_t stats_scratch_for(const mtdao_config& c) {
  size_t a, b;
  return stats_scratch_doubles(c, &a, &b) * sizeof(double);
}

int launch_blocks(int64_t n) {
  int64_t b = (n + kBlock - 1) / kBlock;
  if (b < 1) b = 1;
  if (b > 65536) b = 65536;
  return (int)b;
}

// Algorithm 4: averaged first moments feed the same step (SGDM only).
void launch_sgdm_averaged_momenta(const mtdao_config& c, StepParams p, int V, uint32_t mask, hipStream_t st) {
  dispatch_step(c, V, [&](auto form, auto n, auto xt, auto gt, auto vw) {
    constexpr int FORM = decltype(form)::value, N = decltype(n)::value, VV = decltype(vw)::value;
    if constexpr (FORM == kSgdm) {
      using XT = typename decltype(xt)::type;
      using GT = typename decltype(gt)::type;
      if (c.replicas > 1 && c.replicas <= kWaveMaxK) {
        // one wavefront per replica, one pass
        const int64_t per = (int64_t)64 * VV;
        p.tiles = (p.P + per - 1) / per;
        hipLaunchKernelGGL((k_sgdm_averaged_momenta_waves<N, XT, GT, VV, kStepNT>), grid_for(p.tiles, 1),
                           dim3(64 * c.replicas), 0, st, p, mask, c.replicas);
        return;
      }
      constexpr int C = piece_for(VV);
      p.tiles = tiles_for<kBlock * VV, C>(p.P);
      hipLaunchKernelGGL((k_sgdm_averaged_momenta<N, XT, GT, VV, kStepNT, C>), grid_for(p.tiles, 1), dim3(kBlock), 0,
                         st, p, mask, c.replicas);
    }
  });
}

}  // namespace

// ===================================================================== ABI

extern "C" {

int32_t mtdao_workspace_bytes(const mtdao_config* cfg, size_t* bytes) {
  const int32_t r = validate(cfg, &g_err);
  if (r != MTDAO_OK) return r;
  if (!bytes) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = workspace_for(*cfg);
  return MTDAO_OK;
}

int32_t mtdao_stats_scratch_bytes(const mtdao_config* cfg, size_t* bytes) {
  const int32_t r = validate(cfg, &g_err);
  if (r != MTDAO_OK) return r;
  if (!bytes) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "bytes is NULL");
  *bytes = stats_scratch_for(*cfg);
  return MTDAO_OK;
}

int32_t mtdao_schedule(const mtdao_config* cfg, int64_t s, uint32_t* mask) {
  const int32_t r = validate(cfg, &g_err);
  if (r != MTDAO_OK) return r;
  if (!mask) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "mask is NULL");
  if (s < 1) return fail(&g_err, MTDAO_ERR_RANGE, "step %lld < 1", (long long)s);
  *mask = schedule_mask(*cfg, s);
  return MTDAO_OK;
}

int32_t mtdao_init(const mtdao_config* cfg, const mtdao_buffers* bufs, void* workspace, size_t workspace_bytes,
                   void* hip_stream, mtdao_handle** out) {
  int32_t r = validate(cfg, &g_err);
  if (r != MTDAO_OK) return r;
  if (!bufs || !out) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "bufs or out is NULL");
  const mtdao_config& c = *cfg;
  const int64_t KP = (int64_t)c.replicas * c.numel;
  const int N = c.n_moments;
  // device pointers and their extents
  std::vector<std::pair<const void*, int64_t>> ranges;
  if (c.numel > 0) {
    if (!bufs->x) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "x is NULL");
    ranges.push_back({bufs->x, KP * esize(c.param_dtype)});
    for (int j = 0; j < N; ++j) {
      if (!bufs->u[j]) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "u[%d] is NULL", j);
      ranges.push_back({bufs->u[j], KP * 4});
    }
    if (has_v(c)) {
      if (!bufs->v) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "v is NULL (Adam and ADOPT need it)");
      ranges.push_back({bufs->v, KP * 4});
    }
    if (c.outer_opt == MTDAO_OUTER_NESTEROV) {
      if (!bufs->x_outer || !bufs->x_outer_mom)
        return fail(&g_err, MTDAO_ERR_INVALID_ARG, "x_outer / x_outer_mom are NULL (Nesterov OuterOpt needs them)");
      ranges.push_back({bufs->x_outer, c.numel * 4});
      ranges.push_back({bufs->x_outer_mom, c.numel * 4});
    }
    for (auto& rg : ranges)
      if (!aligned16(rg.first)) return fail(&g_err, MTDAO_ERR_ALIGN, "a state buffer is not 16-byte aligned");
    for (size_t a = 0; a < ranges.size(); ++a)
      for (size_t b = a + 1; b < ranges.size(); ++b)
        if (overlap(ranges[a].first, ranges[a].second, ranges[b].first, ranges[b].second))
          return fail(&g_err, MTDAO_ERR_INVALID_ARG, "state buffers overlap");
  }
  const size_t need = workspace_for(c);
  if (need > 0) {
    if (!workspace) return fail(&g_err, MTDAO_ERR_WORKSPACE, "workspace of %zu bytes required", need);
    if (workspace_bytes < need)
      return fail(&g_err, MTDAO_ERR_WORKSPACE, "workspace %zu bytes < required %zu", workspace_bytes, need);
    if ((reinterpret_cast<uintptr_t>(workspace) & 255u) != 0)
      return fail(&g_err, MTDAO_ERR_ALIGN, "workspace is not 256-byte aligned");
  }

  mtdao_handle* h = new mtdao_handle();
  h->cfg = c;
  if (c.n_tensors > 0) h->tensors.assign(c.tensor_numel, c.tensor_numel + c.n_tensors);
  else h->tensors.assign(1, c.numel);
  h->cfg.n_tensors = (int32_t)h->tensors.size();
  h->cfg.tensor_numel = h->tensors.data();
  h->x = bufs->x;
  for (int j = 0; j < N; ++j) h->u[j] = bufs->u[j];
  h->v = has_v(c) ? bufs->v : nullptr;
  if (c.outer_opt == MTDAO_OUTER_NESTEROV) {
    h->x_outer = bufs->x_outer;
    h->x_outer_mom = bufs->x_outer_mom;
  }
  h->s = c.start_step;
  if (need > 0) {
    const size_t scale_bytes = ((size_t)c.replicas * sizeof(float) + 255) / 256 * 256;
    h->scale = reinterpret_cast<float*>(workspace);
    h->partials = reinterpret_cast<double*>(reinterpret_cast<char*>(workspace) + scale_bytes);
    h->norm_blocks = norm_blocks_for(c.numel);
  }

  hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
  if (!bufs->init_states && c.numel > 0) {
    const int nb = launch_blocks(c.numel);
    if (c.replicas > 1) {
      if (c.param_dtype == MTDAO_F32)
        hipLaunchKernelGGL(k_broadcast_row0<float>, dim3(nb), dim3(kBlock), 0, st, (float*)h->x, c.numel, c.replicas);
      else
        hipLaunchKernelGGL(k_broadcast_row0<uint16_t>, dim3(nb), dim3(kBlock), 0, st, (uint16_t*)h->x, c.numel,
                           c.replicas);
    }
    const int zb = launch_blocks(KP);
    for (int j = 0; j < N; ++j) hipLaunchKernelGGL(k_fill_zero, dim3(zb), dim3(kBlock), 0, st, h->u[j], KP);
    if (h->v) hipLaunchKernelGGL(k_fill_zero, dim3(zb), dim3(kBlock), 0, st, h->v, KP);
    if (h->x_outer) {
      if (c.param_dtype == MTDAO_F32)
        hipLaunchKernelGGL(k_row0_to_f32<float>, dim3(nb), dim3(kBlock), 0, st, (const float*)h->x, h->x_outer, c.numel);
      else
        hipLaunchKernelGGL(k_row0_to_f32<uint16_t>, dim3(nb), dim3(kBlock), 0, st, (const uint16_t*)h->x, h->x_outer,
                           c.numel);
      hipLaunchKernelGGL(k_fill_zero, dim3(nb), dim3(kBlock), 0, st, h->x_outer_mom, c.numel);
    }
    r = hip_check(&g_err, hipGetLastError(), "mtdao_init launch");
    if (r != MTDAO_OK) {
      delete h;
      return r;
    }
  }
  g_err.clear();
  *out = h;
  return MTDAO_OK;
}

}  // extern "C"

namespace {

int32_t check_step_args(mtdao_handle* h, const void* grads, float lr, float adopt_clip) {
  const mtdao_config& c = h->cfg;
  const int64_t P = c.numel, KP = (int64_t)c.replicas * P;
  if (!std::isfinite(lr)) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "lr is not finite");
  if (!std::isfinite(adopt_clip)) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "adopt_clip is not finite");
  if (P > 0) {
    if (!grads) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "grads is NULL");
    if (!aligned16(grads)) return fail(&h->err, MTDAO_ERR_ALIGN, "grads is not 16-byte aligned");
    const int64_t gb = KP * esize(c.grad_dtype);
    bool ov = overlap(grads, gb, h->x, KP * esize(c.param_dtype));
    for (int j = 0; j < c.n_moments; ++j) ov = ov || overlap(grads, gb, h->u[j], KP * 4);
    if (h->v) ov = ov || overlap(grads, gb, h->v, KP * 4);
    if (h->x_outer) ov = ov || overlap(grads, gb, h->x_outer, P * 4) || overlap(grads, gb, h->x_outer_mom, P * 4);
    if (ov) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "grads overlaps a state buffer");
  }
  return MTDAO_OK;
}

int32_t resolve_mask(mtdao_handle* h, uint32_t mask, int64_t s, uint32_t* out) {
  const mtdao_config& c = h->cfg;
  if (mask == MTDAO_SYNC_AUTO) {
    *out = s >= 1 ? schedule_mask(c, s) : 0u;
    return MTDAO_OK;
  }
  if (mask & ~valid_bits(c))
    return fail(&h->err, MTDAO_ERR_INVALID_ARG, "mask 0x%x has bits beyond the %d states", mask,
                1 + c.n_moments + (has_v(c) ? 1 : 0));
  *out = mask;
  return MTDAO_OK;
}

OuterParams outer_params(const mtdao_handle* h, bool update = true) {
  OuterParams o;
  o.xo = h->x_outer;
  o.mom = h->x_outer_mom;
  o.lr = h->cfg.outer_lr;
  o.mu = h->cfg.outer_momentum;
  o.update = update ? 1 : 0;
  return o;
}

// The Nesterov outer step runs at most once per step s: an averaging of x
// that repeats the one of this s (mtdao_sync after mtdao_step_sync, a second
// mtdao_sync or mtdao_sync_stats) only averages rows that are already equal.
// Returns whether the outer step is to run now and records it.
bool claim_outer_step(mtdao_handle* h, uint32_t work, int64_t s) {
  if (!h->x_outer || !(work & 1u)) return false;
  if (h->outer_done_s == s) return false;
  h->outer_done_s = s;
  return true;
}

BiasCorrection bias_correction_of(const mtdao_config& c) {
  BiasCorrection b;
  std::memset(&b, 0, sizeof b);
  for (int j = 0; j < c.n_moments; ++j) {
    b.beta[j] = c.beta1[j];
    b.omega[j] = c.omega[j];
  }
  b.beta2 = c.beta2;
  b.n = c.n_moments;
  b.on = (c.form == MTDAO_ADAM && c.bias_correction) ? 1 : 0;
  return b;
}

// Where a launch takes its update number from on the device.
struct DeviceSource {
  const DeviceStep* dev = nullptr;
  int64_t k = 0;
  const float* lr_table = nullptr;
  const float* clip_table = nullptr;
  int64_t len = 0;
};

// Per-step scalars of update s in double, rounded once to fp32; launches
// the clip-norm reduction first when the configuration clips.  With a
// device source the kernels form lr, the ADOPT clip and the bias-corrected
// weights from the device-side update number instead.
StepParams prepare_step(mtdao_handle* h, const void* grads, float lr, float adopt_clip, int64_t s, hipStream_t st,
                        const DeviceSource& ds = DeviceSource()) {
  const mtdao_config& c = h->cfg;
  const int64_t P = c.numel;
  StepParams p;
  std::memset(&p, 0, sizeof p);
  p.x = h->x;
  p.g = grads;
  for (int j = 0; j < c.n_moments; ++j) p.u[j] = h->u[j];
  p.v = h->v;
  p.P = P;
  p.replicas = c.replicas;
  double wsum = 0.0;
  for (int j = 0; j < c.n_moments; ++j) {
    p.beta[j] = c.beta1[j];
    p.omb[j] = (float)(1.0 - (double)c.beta1[j]);
    wsum += (double)c.omega[j];
  }
  step_scalars(bias_correction_of(c), s, p.w, &p.inv_bc2);
  p.gw = (float)(1.0 - wsum);
  p.beta2 = c.beta2;
  p.omb2 = (float)(1.0 - (double)c.beta2);
  p.eps = c.eps;
  p.dev = ds.dev;
  p.dev_k = ds.k;
  p.lr_table = ds.lr_table;
  p.clip_table = ds.clip_table;
  p.table_len = ds.len;
  p.bc = bias_correction_of(c);
  p.lr = lr;
  p.clip = adopt_clip;
  p.scale = nullptr;
  p.outer = outer_params(h);
  if (c.form != MTDAO_ADOPT && c.clip_rho > 0.0f) {
    const int Vg = (P % 4 == 0) ? 4 : 1;  // 16-byte (fp32) or 8-byte (bf16) slots
    if (c.grad_dtype == MTDAO_F32) launch_norm<float>(grads, P, c.replicas, Vg, h->norm_blocks, h->partials, st);
    else launch_norm<uint16_t>(grads, P, c.replicas, Vg, h->norm_blocks, h->partials, st);
    hipLaunchKernelGGL(k_clip_finalize, dim3(c.replicas), dim3(kFinalizeBlock), 0, st, h->partials, h->norm_blocks,
                       (double)c.clip_rho, h->scale);
    p.scale = h->scale;
  }
  return p;
}

// One vector width for every buffer the step touches: 4 elements when every
// row start keeps 16-byte (fp32) and 8-byte (bf16) alignment, else 1.
int step_vec_width(const mtdao_config& c) { return (c.numel % 4 == 0) ? 4 : 1; }

bool adopt_first_update(const mtdao_config& c, int64_t s) {
  return c.form == MTDAO_ADOPT && c.adopt_order == MTDAO_ADOPT_PREV && s == 1;
}

void launch_adopt_first(mtdao_handle* h, const void* grads, hipStream_t st) {
  const mtdao_config& c = h->cfg;
  const int Vi = (c.numel % 4 == 0) ? 4 : 1;
  if (c.grad_dtype == MTDAO_F32) launch_adopt_init<float>(grads, h->v, c.numel, c.replicas, Vi, st);
  else launch_adopt_init<uint16_t>(grads, h->v, c.numel, c.replicas, Vi, st);
}

void launch_means(mtdao_handle* h, uint32_t m, bool outer_update, hipStream_t st) {
  const mtdao_config& c = h->cfg;
  MeanParams mp;
  std::memset(&mp, 0, sizeof mp);
  mp.P = c.numel;
  mp.K = c.replicas;
  mp.outer_state = -1;
  mp.outer = outer_params(h);
  // fp32 moment states (and fp32 x) in one launch, bf16 x in its own
  int n = 0;
  if ((m & 1u) && c.param_dtype == MTDAO_F32) {
    if (outer_update) mp.outer_state = n;
    mp.state[n++] = h->x;
  }
  for (int j = 0; j < c.n_moments; ++j)
    if (m & (1u << (j + 1))) mp.state[n++] = h->u[j];
  if (h->v && (m & (1u << (c.n_moments + 1)))) mp.state[n++] = h->v;
  if (n > 0) launch_mean<float>(mp, n, vec_width(MTDAO_F32, c.numel), st);
  if ((m & 1u) && c.param_dtype == MTDAO_BF16) {
    MeanParams xp = mp;
    xp.state[0] = h->x;
    xp.outer_state = outer_update ? 0 : -1;
    launch_mean<uint16_t>(xp, 1, vec_width(MTDAO_BF16, c.numel), st);
  }
}

// mtdao_step_sync after its argument checks; with a device source the
// kernels form their step-dependent scalars from the device-side update
// number.
int32_t step_sync_launch(mtdao_handle* h, const void* grads, float lr, float adopt_clip, uint32_t mask,
                         uint32_t* applied_mask, hipStream_t st, const DeviceSource& ds) {
  const int64_t s = h->s + 1;
  const RoctxRange range("%s s=%lld mask=0x%x", ds.dev ? "mtdao_step_sync_device" : "mtdao_step_sync", (long long)s, mask);
  uint32_t m;
  int32_t r = resolve_mask(h, mask, s, &m);
  if (r != MTDAO_OK) return r;
  h->s = s;
  if (applied_mask) *applied_mask = m;
  const mtdao_config& c = h->cfg;
  if (c.numel == 0) return MTDAO_OK;
  const StepParams p = prepare_step(h, grads, lr, adopt_clip, s, st, ds);
  // s is new, so an outer step due here has not run yet
  const bool outer_update = claim_outer_step(h, m, s);
  // K = 1: the mean is the row; only an outer step on x still has work
  const uint32_t work = c.replicas > 1 ? m : (outer_update ? 1u : 0u);
  if (adopt_first_update(c, s)) {
    launch_adopt_first(h, grads, st);
    if (work != 0) launch_means(h, work, outer_update, st);
  } else if (work == 0) {
    launch_step(c, p, step_vec_width(c), st);
  } else if (c.sync_order == MTDAO_SYNC_MOMENTA_IN_STEP && (work & ~1u) != 0) {
    launch_sgdm_averaged_momenta(c, p, step_vec_width(c), work, st);
  } else {
    launch_step_sync(c, p, step_vec_width(c), work, st);
  }
  return hip_check(&h->err, hipGetLastError(), "mtdao_step_sync launch");
}

}  // namespace

extern "C" {

int32_t mtdao_local_step(mtdao_handle* h, const void* grads, float lr, float adopt_clip, void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  const RoctxRange range("mtdao_local_step s=%lld", (long long)(h->s + 1));
  int32_t r = check_step_args(h, grads, lr, adopt_clip);
  if (r != MTDAO_OK) return r;
  const int64_t s = ++h->s;
  if (h->cfg.numel == 0) return MTDAO_OK;
  hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
  const StepParams p = prepare_step(h, grads, lr, adopt_clip, s, st);
  if (adopt_first_update(h->cfg, s)) launch_adopt_first(h, grads, st);
  else launch_step(h->cfg, p, step_vec_width(h->cfg), st);
  return hip_check(&h->err, hipGetLastError(), "mtdao_local_step launch");
}

int32_t mtdao_sync(mtdao_handle* h, uint32_t mask, uint32_t* applied_mask, void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  const RoctxRange range("mtdao_sync s=%lld mask=0x%x", (long long)h->s, mask);
  uint32_t m;
  int32_t r = resolve_mask(h, mask, h->s, &m);
  if (r != MTDAO_OK) return r;
  const mtdao_config& c = h->cfg;
  if (c.sync_order == MTDAO_SYNC_MOMENTA_IN_STEP && (m & ~1u) != 0)
    return fail(&h->err, MTDAO_ERR_INVALID_ARG,
                "with sync_order MOMENTA_IN_STEP the moments are averaged inside mtdao_step_sync (mask 0x%x)", m);
  if (applied_mask) *applied_mask = m;
  if (c.numel == 0) return MTDAO_OK;
  const bool outer_update = claim_outer_step(h, m, h->s);
  // K = 1: the mean is the row; only an outer step on x still has work
  const uint32_t work = c.replicas > 1 ? m : (outer_update ? 1u : 0u);
  if (work == 0) return MTDAO_OK;
  launch_means(h, work, outer_update, reinterpret_cast<hipStream_t>(hip_stream));
  return hip_check(&h->err, hipGetLastError(), "mtdao_sync launch");
}

}  // extern "C"

namespace {

// Device scratch of mtdao_sync_stats_static, for callers that cannot
// allocate device memory: one array per GPU for the life of the process,
// shared by every call on that GPU.  In host code `scratch` only names the
// symbol; its device address comes from hipGetSymbolAddress, once per
// device, with that device current.
constexpr size_t kStaticScratchDoubles = MTDAO_STATIC_SCRATCH_BYTES / sizeof(double);
__device__ __align__(256) double scratch[kStaticScratchDoubles];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
double* g_scratch_ptr[kMaxDevices] = {};

// Device address of this device's `scratch`, looked up on first use.
int32_t static_scratch(mtdao_handle* h, double** out) {
  int dev = -1;
  int32_t r = hip_check(&h->err, hipGetDevice(&dev), "hipGetDevice");
  if (r != MTDAO_OK) return r;
  if (dev < 0 || dev >= kMaxDevices)
    return fail(&h->err, MTDAO_ERR_INVALID_ARG, "device %d outside [0, %d)", dev, kMaxDevices);
  std::lock_guard<std::mutex> lock(g_scratch_mutex);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    r = hip_check(&h->err, hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)), "hipGetSymbolAddress(scratch)");
    if (r != MTDAO_OK) return r;
    if (!p) return fail(&h->err, MTDAO_ERR_HIP, "hipGetSymbolAddress(scratch) gave NULL");
    g_scratch_ptr[dev] = reinterpret_cast<double*>(p);
  }
  *out = g_scratch_ptr[dev];
  return MTDAO_OK;
}

// Checks shared by both diagnostics entry points (before any scratch check).
int32_t check_stats_args(mtdao_handle* h, double* host_stats) {
  const mtdao_config& c = h->cfg;
  if (c.replicas > kStatsMaxK)
    return fail(&h->err, MTDAO_ERR_INVALID_ARG, "diagnostics support up to %d replicas (K=%d)", kStatsMaxK, c.replicas);
  if (!host_stats) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "host_stats is NULL");
  return MTDAO_OK;
}

// mtdao_sync_stats after its scratch checks: the averaging with the
// diagnostics of every averaged state, partial sums in `scratch` (at least
// stats_scratch_for(cfg) bytes, 256-byte aligned; every word the kernels
// read is written first in the same call, so nothing needs clearing), the
// finalized rows copied to host_stats through a buffer on the stack.
int32_t run_sync_stats(mtdao_handle* h, uint32_t mask, uint32_t* applied_mask, double* scratch, double* host_stats,
                       hipStream_t st) {
  const RoctxRange range("mtdao_sync_stats s=%lld mask=0x%x", (long long)h->s, mask);
  const mtdao_config& c = h->cfg;
  uint32_t m;
  int32_t r = resolve_mask(h, mask, h->s, &m);
  if (r != MTDAO_OK) return r;
  if (c.sync_order == MTDAO_SYNC_MOMENTA_IN_STEP && (m & ~1u) != 0)
    return fail(&h->err, MTDAO_ERR_INVALID_ARG,
                "with sync_order MOMENTA_IN_STEP the moments are averaged inside mtdao_step_sync (mask 0x%x)", m);
  if (applied_mask) *applied_mask = m;
  constexpr int nslots = 2 + kMaxN;
  for (int i = 0; i < nslots * kStatsStride; ++i) host_stats[i] = NAN;
  if (m == 0 || c.numel == 0) return MTDAO_OK;
  double* partials = scratch;
  size_t fp32_part, bf16_part;
  stats_scratch_doubles(c, &fp32_part, &bf16_part);
  double* part_x = partials + fp32_part;
  double* out = part_x + bf16_part;  // [2][nslots][stride]
  // state ids of the fp32 launch, in launch order
  int ids[2 + kMaxN];
  MeanParams mp;
  std::memset(&mp, 0, sizeof mp);
  mp.P = c.numel;
  mp.K = c.replicas;
  mp.outer_state = -1;
  // under Nesterov the diagnostics of x are those of the pseudo-gradients
  // x_outer - x^m also when the outer step of this s has already run
  mp.outer = outer_params(h, claim_outer_step(h, m, h->s));
  int n = 0;
  if ((m & 1u) && c.param_dtype == MTDAO_F32) {
    if (h->x_outer) mp.outer_state = n;
    ids[n] = 0;
    mp.state[n++] = h->x;
  }
  for (int j = 0; j < c.n_moments; ++j)
    if (m & (1u << (j + 1))) {
      ids[n] = j + 1;
      mp.state[n++] = h->u[j];
    }
  if (h->v && (m & (1u << (c.n_moments + 1)))) {
    ids[n] = c.n_moments + 1;
    mp.state[n++] = h->v;
  }
  if (n > 0) launch_stats<float>(mp, n, vec_width(MTDAO_F32, c.numel), partials, out, st);
  const bool bf16_x = (m & 1u) && c.param_dtype == MTDAO_BF16;
  if (bf16_x) {
    MeanParams q = mp;
    std::memset(q.state, 0, sizeof q.state);
    q.state[0] = h->x;
    q.outer_state = h->x_outer ? 0 : -1;
    launch_stats<uint16_t>(q, 1, vec_width(MTDAO_BF16, c.numel), part_x, out + nslots * kStatsStride, st);
  }
  r = hip_check(&h->err, hipGetLastError(), "mtdao_sync_stats launch");
  if (r != MTDAO_OK) return r;
  double rows[2 * nslots * kStatsStride];
  r = hip_check(&h->err, hipMemcpyAsync(rows, out, sizeof rows, hipMemcpyDeviceToHost, st), "mtdao_sync_stats copy");
  if (r != MTDAO_OK) return r;
  r = hip_check(&h->err, hipStreamSynchronize(st), "mtdao_sync_stats wait");
  if (r != MTDAO_OK) return r;
  for (int i = 0; i < n; ++i)
    for (int k = 0; k < kStatsStride; ++k) host_stats[ids[i] * kStatsStride + k] = rows[i * kStatsStride + k];
  if (bf16_x)
    for (int k = 0; k < kStatsStride; ++k) host_stats[k] = rows[nslots * kStatsStride + k];
  return MTDAO_OK;
}

}  // namespace

extern "C" {

int32_t mtdao_sync_stats(mtdao_handle* h, uint32_t mask, uint32_t* applied_mask, void* scratch, size_t scratch_bytes,
                         double* host_stats, void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  int32_t r = check_stats_args(h, host_stats);
  if (r != MTDAO_OK) return r;
  const size_t need = stats_scratch_for(h->cfg);
  if (!scratch || scratch_bytes < need)
    return fail(&h->err, MTDAO_ERR_WORKSPACE, "stats scratch of %zu bytes required", need);
  if ((reinterpret_cast<uintptr_t>(scratch) & 255u) != 0)
    return fail(&h->err, MTDAO_ERR_ALIGN, "stats scratch is not 256-byte aligned");
  return run_sync_stats(h, mask, applied_mask, reinterpret_cast<double*>(scratch), host_stats,
                        reinterpret_cast<hipStream_t>(hip_stream));
}

int32_t mtdao_sync_stats_static(mtdao_handle* h, uint32_t mask, uint32_t* applied_mask, double* host_stats,
                                void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  int32_t r = check_stats_args(h, host_stats);
  if (r != MTDAO_OK) return r;
  const size_t need = stats_scratch_for(h->cfg);
  if (need > MTDAO_STATIC_SCRATCH_BYTES)
    return fail(&h->err, MTDAO_ERR_WORKSPACE,
                "the diagnostics of this configuration need %zu bytes of scratch; the static scratch holds %zu "
                "(use mtdao_sync_stats with a caller buffer)",
                need, (size_t)MTDAO_STATIC_SCRATCH_BYTES);
  double* sc = nullptr;
  r = static_scratch(h, &sc);
  if (r != MTDAO_OK) return r;
  return run_sync_stats(h, mask, applied_mask, sc, host_stats, reinterpret_cast<hipStream_t>(hip_stream));
}

int32_t mtdao_step_sync(mtdao_handle* h, const void* grads, float lr, float adopt_clip, uint32_t mask,
                        uint32_t* applied_mask, void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  int32_t r = check_step_args(h, grads, lr, adopt_clip);
  if (r != MTDAO_OK) return r;
  return step_sync_launch(h, grads, lr, adopt_clip, mask, applied_mask, reinterpret_cast<hipStream_t>(hip_stream),
                          DeviceSource());
}

int32_t mtdao_device_step_set(mtdao_handle* h, mtdao_device_step* d, int64_t s, void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  if (!d) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "device step is NULL");
  if (!aligned16(d)) return fail(&h->err, MTDAO_ERR_ALIGN, "device step is not 16-byte aligned");
  if (s < 0) return fail(&h->err, MTDAO_ERR_RANGE, "step %lld < 0", (long long)s);
  int32_t r;
  hipLaunchKernelGGL(k_device_step_set, dim3(1), dim3(64), 0, reinterpret_cast<hipStream_t>(hip_stream),
                     reinterpret_cast<DeviceStep*>(d), s);
  r = hip_check(&h->err, hipGetLastError(), "mtdao_device_step_set launch");
  if (r == MTDAO_OK) h->dev_base = h->s;
  return r;
}

int32_t mtdao_device_step_advance(mtdao_handle* h, mtdao_device_step* d, void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  if (!d) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "device step is NULL");
  if (!aligned16(d)) return fail(&h->err, MTDAO_ERR_ALIGN, "device step is not 16-byte aligned");
  const int64_t n = h->s - h->dev_base;
  if (n == 0) return MTDAO_OK;
  hipLaunchKernelGGL(k_device_step_add, dim3(1), dim3(64), 0, reinterpret_cast<hipStream_t>(hip_stream),
                     reinterpret_cast<DeviceStep*>(d), n);
  const int32_t r = hip_check(&h->err, hipGetLastError(), "mtdao_device_step_advance launch");
  if (r == MTDAO_OK) h->dev_base = h->s;
  return r;
}

int32_t mtdao_step_sync_device(mtdao_handle* h, const void* grads, mtdao_device_step* d, const float* lr_table,
                               const float* clip_table, int64_t table_len, uint32_t mask, uint32_t* applied_mask,
                               void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  int32_t r = check_step_args(h, grads, 0.0f, 0.0f);
  if (r != MTDAO_OK) return r;
  if (!d || !lr_table) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "device step or lr table is NULL");
  if (!aligned16(d)) return fail(&h->err, MTDAO_ERR_ALIGN, "device step is not 16-byte aligned");
  if (table_len < 1) return fail(&h->err, MTDAO_ERR_RANGE, "table_len %lld < 1", (long long)table_len);
  if (adopt_first_update(h->cfg, h->s + 1))
    return fail(&h->err, MTDAO_ERR_INVALID_ARG,
                "ADOPT's first update (v = g^2 only) goes through mtdao_local_step or mtdao_step_sync");
  DeviceSource ds;
  ds.dev = reinterpret_cast<const DeviceStep*>(d);
  ds.k = h->s + 1 - h->dev_base;
  ds.lr_table = lr_table;
  ds.clip_table = clip_table;
  ds.len = table_len;
  return step_sync_launch(h, grads, 0.0f, 0.0f, mask, applied_mask, reinterpret_cast<hipStream_t>(hip_stream), ds);
}

int32_t mtdao_read_state(mtdao_handle* h, int32_t state, int32_t replica, int64_t offset, int64_t count,
                         void* host_dst, void* hip_stream) {
  if (!h) return fail(&g_err, MTDAO_ERR_INVALID_ARG, "handle is NULL");
  const mtdao_config& c = h->cfg;
  const int32_t nstates = 1 + c.n_moments + (has_v(c) ? 1 : 0);
  const bool outer_state = state == MTDAO_STATE_X_OUTER || state == MTDAO_STATE_OUTER_MOM;
  if (outer_state && !h->x_outer)
    return fail(&h->err, MTDAO_ERR_INVALID_ARG, "state %d needs the Nesterov OuterOpt", state);
  if (!outer_state && (state < 0 || state >= nstates))
    return fail(&h->err, MTDAO_ERR_INVALID_ARG, "state %d outside [0, %d)", state, nstates);
  if (replica < 0 || replica >= (outer_state ? 1 : c.replicas))
    return fail(&h->err, MTDAO_ERR_RANGE, "replica %d outside [0, %d)", replica, outer_state ? 1 : c.replicas);
  if (offset < 0 || count < 0 || offset > c.numel || count > c.numel - offset)
    return fail(&h->err, MTDAO_ERR_RANGE, "range [%lld, +%lld) outside [0, %lld)", (long long)offset,
                (long long)count, (long long)c.numel);
  if (count == 0) return MTDAO_OK;
  if (!host_dst) return fail(&h->err, MTDAO_ERR_INVALID_ARG, "host_dst is NULL");
  const void* base;
  int64_t es;
  if (outer_state) {
    base = state == MTDAO_STATE_X_OUTER ? h->x_outer : h->x_outer_mom;
    es = 4;
  } else if (state == 0) {
    base = h->x;
    es = esize(c.param_dtype);
  } else if (state <= c.n_moments) {
    base = h->u[state - 1];
    es = 4;
  } else {
    base = h->v;
    es = 4;
  }
  const char* src = reinterpret_cast<const char*>(base) + ((int64_t)replica * c.numel + offset) * es;
  hipStream_t st = reinterpret_cast<hipStream_t>(hip_stream);
  int32_t r = hip_check(&h->err, hipMemcpyAsync(host_dst, src, (size_t)(count * es), hipMemcpyDeviceToHost, st),
                        "mtdao_read_state copy");
  if (r != MTDAO_OK) return r;
  return hip_check(&h->err, hipStreamSynchronize(st), "mtdao_read_state wait");
}

int64_t mtdao_step_count(const mtdao_handle* h) { return h ? h->s : -1; }

const char* mtdao_last_error(const mtdao_handle* h) { return h ? h->err.c_str() : g_err.c_str(); }

void mtdao_destroy(mtdao_handle* h) { delete h; }

}  // extern "C"
