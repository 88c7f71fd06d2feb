// Device kernels of the MT-DAO hot path for CDNA4 (gfx950).
//
// All kernels are streaming, HBM-bound passes: the local step reads x, g,
// u^1..u^N, v once and writes x, u^1..u^N, v once per element (no MFMA:
// there is no contraction).  Every thread owns V consecutive elements of
// one replica row per vector slot, so loads and stores are 16-byte vector
// accesses and a 64-lane wavefront moves 1 KiB per instruction; all loads
// of a tile are issued before any of them is consumed.  Rows are
// replica-major [K][P].  Two organisations:
//   - one replica row per workgroup (the plain step, the norm pass, the
//     thread-per-column kernels): blockIdx.y is the replica (the state,
//     for the mean), blockIdx.x a tile of the row placed by tile_elem();
//   - one wavefront per replica (the fused step + sync, the mean, the
//     diagnostics and Algorithm 4's step for 1 < K <= 16): a workgroup of
//     K waves takes one piece of 64 V elements of every row, and values
//     that must be averaged meet in LDS.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mtdao {

constexpr int kBlock = 256;
constexpr int kMaxN = 4;
constexpr int kMaxMeanStates = 2 + kMaxN;

enum Form { kAdam = 0, kAdopt = 1, kSgdm = 2 };
enum AdoptOrder { kPrev = 0, kCur = 1 };

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x4 __attribute__((ext_vector_type(4)));
typedef uint16_t u16x8 __attribute__((ext_vector_type(8)));

// ------------------------------------------------------------ conversions

__device__ __forceinline__ float bf16_to_f32(uint16_t b) { return __uint_as_float((uint32_t)b << 16); }

// Round-to-nearest-even fp32 -> bf16 (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return (uint16_t)((u >> 16) | 0x40u);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// A wave-uniform value that no running kernel writes (a parameter table, the
// device-side step count, the clip factors of an earlier launch), read
// through the scalar cache: the load waits only on other scalar loads,
// never on the vector loads of the tile in flight.
template <typename T>
__device__ __forceinline__ T load_uniform(const T* p) {
  return *(const __attribute__((address_space(4))) T*)p;
}

// --------------------------------------------------- vector load / store
//
// load_v<T, V>(p, e, out): V consecutive elements starting at element e,
// widened to fp32.  T = float, or uint16_t holding bf16 bit patterns.  V = 1 (scalar path for rows whose
// length breaks 16-byte alignment), 4 or 8.

template <bool NT, typename VT>
__device__ __forceinline__ VT ld(const VT* p) {
  if constexpr (NT) return __builtin_nontemporal_load(p);
  else return *p;
}

template <bool NT, typename VT>
__device__ __forceinline__ void st(VT* p, VT v) {
  if constexpr (NT) __builtin_nontemporal_store(v, p);
  else *p = v;
}

template <typename T, int V, bool NT>
__device__ __forceinline__ void load_v(const T* __restrict__ p, int64_t e, float (&o)[V]) {
  if constexpr (sizeof(T) == 4) {
    const float* q = reinterpret_cast<const float*>(p) + e;
    if constexpr (V == 1) {
      o[0] = ld<NT>(q);
    } else {
#pragma unroll
      for (int k = 0; k < V / 4; ++k) {
        f32x4 a = ld<NT>(reinterpret_cast<const f32x4*>(q) + k);
        o[4 * k + 0] = a.x; o[4 * k + 1] = a.y; o[4 * k + 2] = a.z; o[4 * k + 3] = a.w;
      }
    }
  } else {
    const uint16_t* q = reinterpret_cast<const uint16_t*>(p) + e;
    if constexpr (V == 1) {
      o[0] = bf16_to_f32(ld<NT>(q));
    } else if constexpr (V == 4) {
      u16x4 a = ld<NT>(reinterpret_cast<const u16x4*>(q));
#pragma unroll
      for (int k = 0; k < 4; ++k) o[k] = bf16_to_f32(a[k]);
    } else {
#pragma unroll
      for (int k = 0; k < V / 8; ++k) {
        u16x8 a = ld<NT>(reinterpret_cast<const u16x8*>(q) + k);
#pragma unroll
        for (int t = 0; t < 8; ++t) o[8 * k + t] = bf16_to_f32(a[t]);
      }
    }
  }
}

template <typename T, int V, bool NT>
__device__ __forceinline__ void store_v(T* __restrict__ p, int64_t e, const float (&o)[V]) {
  if constexpr (sizeof(T) == 4) {
    float* q = reinterpret_cast<float*>(p) + e;
    if constexpr (V == 1) {
      st<NT>(q, o[0]);
    } else {
#pragma unroll
      for (int k = 0; k < V / 4; ++k) {
        f32x4 a = {o[4 * k + 0], o[4 * k + 1], o[4 * k + 2], o[4 * k + 3]};
        st<NT>(reinterpret_cast<f32x4*>(q) + k, a);
      }
    }
  } else {
    uint16_t* q = reinterpret_cast<uint16_t*>(p) + e;
    if constexpr (V == 1) {
      st<NT>(q, f32_to_bf16(o[0]));
    } else if constexpr (V == 4) {
      u16x4 a;
#pragma unroll
      for (int k = 0; k < 4; ++k) a[k] = f32_to_bf16(o[k]);
      st<NT>(reinterpret_cast<u16x4*>(q), a);
    } else {
#pragma unroll
      for (int k = 0; k < V / 8; ++k) {
        u16x8 a;
#pragma unroll
        for (int t = 0; t < 8; ++t) a[t] = f32_to_bf16(o[8 * k + t]);
        st<NT>(reinterpret_cast<u16x8*>(q) + k, a);
      }
    }
  }
}

// ------------------------------------------------------ tile -> elements
//
// Workgroups are dispatched round-robin over the 8 XCDs, so with a plain
// tile sequence XCD i works on tiles i, i + 8, ...  The HBM rate of a
// streaming pass depends on how large a contiguous piece each XCD takes in
// turn: pieces of 512 B - 1 KiB per stream spread the XCDs' traffic over
// the memory channels best, 2 KiB pieces worst (about 10 % apart on MI355X
// for the same bytes).  tile_elem() therefore splits a tile of B*V*U
// elements into pieces of C elements and places piece j of tile t at piece
// index ((t / 8) * R + j) * 8 + t % 8 of the row (R = pieces per tile), so
// workgroups on one XCD still take one piece in eight and the pieces of a
// tile are 8 C elements apart.  C = 0 keeps the tile contiguous.  Every
// element of the row belongs to exactly one (tile, slot, thread) for
// tiles < tiles_for<B * V * U, C>(P); elements past P are skipped by the
// callers' bounds checks.
template <int T, int C>
__device__ __forceinline__ int64_t tile_elem(int64_t tile, int local) {
  if constexpr (C == 0) {
    return tile * (int64_t)T + local;
  } else {
    static_assert(T % C == 0, "a tile holds whole pieces");
    constexpr int R = T / C;
    const int64_t piece = ((tile >> 3) * R + local / C) * 8 + (tile & 7);
    return piece * C + local % C;
  }
}

// Number of tiles that cover a row of P elements under tile_elem<T, C>.
template <int T, int C>
__host__ __device__ constexpr int64_t tiles_for(int64_t P) {
  if constexpr (C == 0) {
    return (P + T - 1) / T;
  } else {
    const int64_t pieces = (P + C - 1) / C;
    const int64_t per8 = 8 * (int64_t)(T / C);  // pieces covered by 8 consecutive tiles
    return (pieces + per8 - 1) / per8 * 8;
  }
}

// ------------------------------------------------------------ OuterOpt

// Nesterov OuterOpt at an averaging event of x (xo == nullptr: plain
// averaging).  xo, mom: fp32 [P] outer parameters and outer momentum.
struct OuterParams {
  float* xo;
  float* mom;
  float lr;        // outer learning rate
  float mu;        // outer momentum
  int32_t update;  // 0: xo and mom are only read (the outer step of this s already ran)
};

// xbar (the workers' mean) becomes the value every worker restarts from:
// d = xo - xbar; mom = mu mom + d; xo = xo - lr (d + mu mom).
template <int V>
__device__ __forceinline__ void outer_step(const OuterParams& o, int64_t e, float (&xbar)[V]) {
#pragma clang fp contract(off)
  if (o.xo == nullptr || !o.update) return;
  float xo[V], b[V];
  load_v<float, V, false>(o.xo, e, xo);
  load_v<float, V, false>(o.mom, e, b);
#pragma unroll
  for (int t = 0; t < V; ++t) {
    const float d = xo[t] - xbar[t];
    b[t] = __builtin_fmaf(o.mu, b[t], d);
    xo[t] = __builtin_fmaf(-o.lr, __builtin_fmaf(o.mu, b[t], d), xo[t]);
    xbar[t] = xo[t];
  }
  store_v<float, V, false>(o.xo, e, xo);
  store_v<float, V, false>(o.mom, e, b);
}

// The OuterOpt over one piece of 64 V elements whose means sit in LDS,
// means[t * 64 + l] = element l V + t of the piece starting at element e0
// (the layout of the wave-per-replica kernels).  Wave m of the K takes
// every K-th run of 64 consecutive elements, so the fp32 outer parameters
// and momentum are read and written in accesses that are contiguous across
// the lanes of a wave (the column-by-wave order of the mean phase would
// put them 16 bytes apart).  Each element gets exactly outer_step's update.
template <int V>
__device__ __forceinline__ void outer_step_piece(const OuterParams& o, int64_t e0, int64_t P, int32_t K, int32_t m,
                                                 int32_t lane, float* means) {
  for (int j = m * 64 + lane; j < 64 * V; j += 64 * K) {
    if (e0 + j >= P) continue;
    const int l = j / V, t = j % V;
    float a[1] = {means[t * 64 + l]};
    outer_step<1>(o, e0 + j, a);
    means[t * 64 + l] = a[0];
  }
}

// ------------------------------------------------------------ local step

enum StepWindows { kWinOne = 0, kWinHalves = 1, kWinPairs = 2 };

// The update count kept on the device for graph replay (the layout of
// mtdao_device_step): a launch at offset k after the last advance takes
// update s = s + k; k_device_step_add moves s on by a window of calls.
struct DeviceStep {
  int64_t s;
  int64_t reserved;
};

// b^s for s >= 0 by repeated squaring in plain IEEE double multiplies, so
// host and device code compute the same bits.
__host__ __device__ inline double pow_steps(double b, int64_t s) {
#pragma clang fp contract(off)
  double r = 1.0, a = b;
  while (s > 0) {
    if (s & 1) r = r * a;
    a = a * a;
    s >>= 1;
  }
  return r;
}

// Hyper-parameters the step-dependent scalars are formed from.
struct BiasCorrection {
  float beta[kMaxN];
  float omega[kMaxN];
  float beta2;
  int32_t n;
  int32_t on;  // Adam with bias correction
};

// w_j = omega_j / (1 - beta_j^s) and 1 / (1 - beta_2^s) (omega_j and 1
// without correction) in double, rounded once to fp32; the same code on
// the host (eager calls) and in the kernels (device-side s).
__host__ __device__ inline void step_scalars(const BiasCorrection& c, int64_t s, float* w, float* inv_bc2) {
#pragma clang fp contract(off)
  for (int j = 0; j < c.n; ++j)
    w[j] = (float)(c.on ? (double)c.omega[j] / (1.0 - pow_steps((double)c.beta[j], s)) : (double)c.omega[j]);
  *inv_bc2 = (float)(c.on ? 1.0 / (1.0 - pow_steps((double)c.beta2, s)) : 1.0);
}

__global__ __launch_bounds__(64) void k_device_step_set(DeviceStep* __restrict__ d, int64_t s) {
  if (threadIdx.x == 0) d->s = s;
}

__global__ __launch_bounds__(64) void k_device_step_add(DeviceStep* __restrict__ d, int64_t n) {
  if (threadIdx.x == 0) d->s = d->s + n;
}

// Per-launch scalars, prepared on the host in double and rounded to fp32.
struct StepParams {
  void* x;                 // [K][P] params (XT)
  const void* g;           // [K][P] gradients (GT)
  float* u[kMaxN];         // [K][P] first moments
  float* v;                // [K][P] second moment (Adam, ADOPT)
  const float* scale;      // [K] global-norm clip factors, or nullptr
  int64_t P;               // row length
  int64_t tiles;           // tiles of one row (all windows)
  int64_t wlen;            // k_local_step, kWinHalves: elements of the first window
  int32_t replicas;        // K
  float beta[kMaxN];       // beta_{1,j}
  float omb[kMaxN];        // 1 - beta_{1,j}
  float w[kMaxN];          // omega_j (times 1/(1 - beta_{1,j}^s) for bias-corrected Adam)
  float gw;                // 1 - sum_j omega_j: weight of the current gradient
  float beta2, omb2;       // beta_2, 1 - beta_2
  float inv_bc2;           // 1/(1 - beta_2^s) (Adam with bias correction), else 1
  float eps;
  float lr;                // eta_t
  float clip;              // ADOPT c_t (<= 0: no clamp)
  OuterParams outer;       // OuterOpt applied when x is averaged
  // device-side update number (graph replay): when dev is non-null the
  // update is s = dev->s + dev_k, and lr, clip, w and inv_bc2 are formed
  // from it: eta_t = lr_table[s - 1], c_t = clip_table[s - 1] (the last
  // entries beyond table_len; clip off without a table), corrections from bc
  const DeviceStep* dev;
  int64_t dev_k;
  const float* lr_table;
  const float* clip_table;
  int64_t table_len;
  BiasCorrection bc;
};

// A value every lane of the wave holds, moved to a scalar register (the
// fp64 arithmetic below runs in the vector ALU, whose results would
// otherwise each hold a vector register for the rest of the kernel).
__device__ __forceinline__ float wave_uniform(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(int, v)));
}

// The launch's scalars: those of the argument block, or those of the
// device-side update number when it is given (every workgroup forms them;
// a few dozen double multiplies).  Called where every lane of the wave is
// active.
__device__ __forceinline__ StepParams device_scalars(const StepParams& p0) {
#pragma clang fp contract(off)
  if (p0.dev == nullptr) return p0;
  StepParams p = p0;
  const int64_t s = load_uniform(&p0.dev->s) + p0.dev_k;
  const int64_t i = (s < p0.table_len ? s : p0.table_len) - 1;
  p.lr = load_uniform(p0.lr_table + i);
  p.clip = p0.clip_table != nullptr ? load_uniform(p0.clip_table + i) : 0.0f;
  // step_scalars with the moment loop unrolled (a runtime-indexed store
  // would put the whole parameter block in private memory)
#pragma unroll
  for (int j = 0; j < kMaxN; ++j)
    if (j < p0.bc.n)
      p.w[j] = wave_uniform((float)(p0.bc.on ? (double)p0.bc.omega[j] / (1.0 - pow_steps((double)p0.bc.beta[j], s))
                                             : (double)p0.bc.omega[j]));
  p.inv_bc2 = wave_uniform((float)(p0.bc.on ? 1.0 / (1.0 - pow_steps((double)p0.bc.beta2, s)) : 1.0));
  return p;
}

// The update of one element of one replica (the loop body of Algorithm 1, 2
// or 3).  x, u[0..N), v hold the stored values on entry and the updated
// values on exit; graw is the stored gradient and sc the replica's clip
// factor.  Contraction is pinned (explicit fma, no implicit fusion) so
// every kernel that calls this computes bit-identical values.
template <int FORM, int N, int ORDER>
__device__ __forceinline__ void update_element(const StepParams& p, float sc, float graw, float& x,
                                               float (&u)[N], float& v) {
#pragma clang fp contract(off)
  if constexpr (FORM == kAdam) {
    const float gh = sc * graw;
    float num = p.gw * gh;
#pragma unroll
    for (int j = 0; j < N; ++j) {
      u[j] = __builtin_fmaf(p.beta[j], u[j], p.omb[j] * gh);
      num = __builtin_fmaf(p.w[j], u[j], num);
    }
    v = __builtin_fmaf(p.beta2, v, p.omb2 * (gh * gh));
    const float den = __builtin_sqrtf(v * p.inv_bc2) + p.eps;
    x = __builtin_fmaf(-p.lr, num / den, x);
  } else if constexpr (FORM == kAdopt) {
    float gn;
    if constexpr (ORDER == kPrev) {
      gn = graw / (__builtin_sqrtf(v) + p.eps);
      v = __builtin_fmaf(p.beta2, v, p.omb2 * (graw * graw));
    } else {
      v = __builtin_fmaf(p.beta2, v, p.omb2 * (graw * graw));
      gn = graw / (__builtin_sqrtf(v) + p.eps);
    }
    if (p.clip > 0.0f) gn = gn > p.clip ? p.clip : (gn < -p.clip ? -p.clip : gn);
    float delta = p.gw * gn;
#pragma unroll
    for (int j = 0; j < N; ++j) {
      u[j] = __builtin_fmaf(p.beta[j], u[j], p.omb[j] * gn);
      delta = __builtin_fmaf(p.w[j], u[j], delta);
    }
    x = __builtin_fmaf(-p.lr, delta, x);
  } else {
    const float gh = sc * graw;
    float delta = p.gw * gh;
#pragma unroll
    for (int j = 0; j < N; ++j) {
      u[j] = __builtin_fmaf(p.beta[j], u[j], p.omb[j] * gh);
      delta = __builtin_fmaf(p.w[j], u[j], delta);
    }
    x = __builtin_fmaf(-p.lr, delta, x);
  }
}

// One update of all elements of all replicas (Algorithm 1, 2 or 3 body).
//   FORM       kAdam / kAdopt / kSgdm
//   N          number of first moments
//   XT, GT     storage of params / gradients (float or bf16)
//   V, U       elements per vector slot, slots per thread per tile
//   NTM        bit 0: nontemporal loads, bit 1: nontemporal stores
//   ORDER      ADOPT normalisation order (kPrev: v from before this step)
//   B          threads per block
//   C          elements per piece of the tile -> element map (tile_elem)
//   WIN        which rows and ranges a workgroup's tiles cover:
//              kWinOne       blockIdx.y = replica, tiles of the whole row;
//              kWinHalves    blockIdx.y = replica, even workgroups take
//                            [0, wlen) and odd ones [wlen, P);
//              kWinPairs     blockIdx.y = m < ceil(K / 2), even workgroups
//                            take row m and odd ones row m + ceil(K / 2).
//              Each stream is then read at two places at once, half a row
//              or half the replicas apart; measured on MI355X at 1.31B x 4
//              (bare streams, same buffers): 79.5% of the HBM peak for one
//              window, 80.0% for halves, 80.4% for replica pairs.
template <int FORM, int N, typename XT, typename GT, int V, int U, int NTM, int ORDER, int B = kBlock, int C = 0,
          int WIN = kWinOne>
__global__ __launch_bounds__(B) void k_local_step(StepParams p0) {
  constexpr bool NTL = (NTM & 1) != 0, NTS = (NTM & 2) != 0;

  for (int64_t tile = blockIdx.x; tile < p0.tiles; tile += gridDim.x) {
    // the row m and the range [base, end) of it that this tile belongs to
    const int64_t w = WIN == kWinOne ? 0 : (tile & 1);
    const int64_t wt = WIN == kWinOne ? tile : (tile >> 1);
    int64_t m = blockIdx.y, base = 0, end = p0.P;
    if constexpr (WIN == kWinHalves) {
      base = w * p0.wlen;
      end = w == 0 ? p0.wlen : p0.P;
    } else if constexpr (WIN == kWinPairs) {
      m += w * (int64_t)gridDim.y;
      if (m >= p0.replicas) continue;  // odd K: the last row has no partner
    }
    const int64_t row = m * p0.P;
    XT* __restrict__ x = reinterpret_cast<XT*>(p0.x) + row;
    const GT* __restrict__ g = reinterpret_cast<const GT*>(p0.g) + row;
    float* __restrict__ u[N];
#pragma unroll
    for (int j = 0; j < N; ++j) u[j] = p0.u[j] + row;
    float* __restrict__ v = (FORM == kSgdm) ? nullptr : p0.v + row;
    const float sc = (FORM != kAdopt && p0.scale != nullptr) ? load_uniform(p0.scale + m) : 1.0f;
    float gv[U][V], xv[U][V], uv[U][N][V], vv[U][V];
    // issue every load of the tile before any arithmetic
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t e = base + tile_elem<B * V * U, C>(wt, (k * B + (int)threadIdx.x) * V);
      if (e < end) {
        load_v<GT, V, NTL>(g, e, gv[k]);
        load_v<XT, V, NTL>(x, e, xv[k]);
#pragma unroll
        for (int j = 0; j < N; ++j) load_v<float, V, NTL>(u[j], e, uv[k][j]);
        if constexpr (FORM != kSgdm) load_v<float, V, NTL>(v, e, vv[k]);
      }
    }
    // the step-dependent scalars after the loads are in flight (from the
    // device-side update number when there is one)
    const StepParams p = device_scalars(p0);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t e = base + tile_elem<B * V * U, C>(wt, (k * B + (int)threadIdx.x) * V);
      if (e >= end) continue;
#pragma unroll
      for (int t = 0; t < V; ++t) {
        float uu[N];
#pragma unroll
        for (int j = 0; j < N; ++j) uu[j] = uv[k][j][t];
        float vt = (FORM != kSgdm) ? vv[k][t] : 0.0f;
        update_element<FORM, N, ORDER>(p, sc, gv[k][t], xv[k][t], uu, vt);
#pragma unroll
        for (int j = 0; j < N; ++j) uv[k][j][t] = uu[j];
        if constexpr (FORM != kSgdm) vv[k][t] = vt;
      }
      store_v<XT, V, NTS>(x, e, xv[k]);
#pragma unroll
      for (int j = 0; j < N; ++j) store_v<float, V, NTS>(u[j], e, uv[k][j]);
      if constexpr (FORM != kSgdm) store_v<float, V, NTS>(v, e, vv[k]);
    }
  }
}

// Value a state holds once stored: bf16 parameters are rounded.
template <typename T>
__device__ __forceinline__ float as_stored(float a) {
  if constexpr (sizeof(T) == 2) return bf16_to_f32(f32_to_bf16(a));
  else return a;
}

// The replica mean of one element, shared by every averaging kernel:
// S^0 + (sum_{m>=1} (S^m - S^0)) / K, the differences summed in fp64 in
// replica order and the result rounded to fp32 once.  (An fp32 running sum
// loses up to about (K - 1) 2^-24 of the rows' spread, which at large K is
// more than the mean itself carries when the rows nearly cancel.)  Identical
// rows give S^0 back exactly.  rk = 1 / K in fp64.
__device__ __forceinline__ void mean_add(double& d, float a, float s0) { d += (double)a - (double)s0; }
__device__ __forceinline__ float mean_of(float s0, double d, double rk) {
  return (float)__builtin_fma(d, rk, (double)s0);
}

// Local update of every replica followed by the replica mean of the states
// in `mask` (bit 0 = x, bit j = u^j, bit N+1 = v), in one pass.  A thread
// owns V columns of every replica: it updates replica 0..K-1 in order,
// stores the states that are not due, and accumulates the due ones as
// S^0 + (sum_{m>=1} (S^m - S^0)) / K from their stored values -- the same
// arithmetic, in the same order, as k_local_step followed by
// k_replica_mean, so both paths give bit-identical results -- then writes
// that mean to all K rows.  The separate mean pass (2 K sizeof(T) bytes
// per element per due state) disappears.
template <int FORM, int N, typename XT, typename GT, int V, int NTM, int ORDER, int C = 0>
__global__ __launch_bounds__(kBlock) void k_local_step_sync(StepParams p0, uint32_t mask, int32_t K) {
  const StepParams p = device_scalars(p0);
  constexpr bool NTL = (NTM & 1) != 0, NTS = (NTM & 2) != 0;
  const bool sync_x = (mask & 1u) != 0;
  bool sync_u[N];
#pragma unroll
  for (int j = 0; j < N; ++j) sync_u[j] = ((mask >> (j + 1)) & 1u) != 0;
  const bool sync_v = FORM != kSgdm && ((mask >> (N + 1)) & 1u) != 0;
  XT* __restrict__ x = reinterpret_cast<XT*>(p.x);
  const GT* __restrict__ g = reinterpret_cast<const GT*>(p.g);
  const double rk = 1.0 / (double)K;

  for (int64_t tile = blockIdx.x; tile < p.tiles; tile += gridDim.x) {
    const int64_t e = tile_elem<kBlock * V, C>(tile, (int)threadIdx.x * V);
    if (e >= p.P) continue;
    float x0[V], u0[N][V], v0[V];
    double dx[V], du[N][V], dv[V];
#pragma unroll
    for (int t = 0; t < V; ++t) {
      dx[t] = 0.0;
      dv[t] = 0.0;
#pragma unroll
      for (int j = 0; j < N; ++j) du[j][t] = 0.0;
    }
    for (int32_t m = 0; m < K; ++m) {
      const int64_t r = (int64_t)m * p.P + e;
      float gv[V], xv[V], uv[N][V], vv[V];
      load_v<GT, V, NTL>(g, r, gv);
      load_v<XT, V, NTL>(x, r, xv);
#pragma unroll
      for (int j = 0; j < N; ++j) load_v<float, V, NTL>(p.u[j], r, uv[j]);
      if constexpr (FORM != kSgdm) load_v<float, V, NTL>(p.v, r, vv);
      const float sc = (FORM != kAdopt && p.scale != nullptr) ? load_uniform(p.scale + m) : 1.0f;
#pragma unroll
      for (int t = 0; t < V; ++t) {
        float uu[N];
#pragma unroll
        for (int j = 0; j < N; ++j) uu[j] = uv[j][t];
        float vt = (FORM != kSgdm) ? vv[t] : 0.0f;
        update_element<FORM, N, ORDER>(p, sc, gv[t], xv[t], uu, vt);
        xv[t] = as_stored<XT>(xv[t]);
#pragma unroll
        for (int j = 0; j < N; ++j) uv[j][t] = uu[j];
        vv[t] = vt;
      }
      // states not due: store now; due: accumulate the shifted sum
      if (sync_x) {
#pragma unroll
        for (int t = 0; t < V; ++t) {
          if (m == 0) x0[t] = xv[t];
          else mean_add(dx[t], xv[t], x0[t]);
        }
      } else {
        store_v<XT, V, NTS>(x, r, xv);
      }
#pragma unroll
      for (int j = 0; j < N; ++j) {
        if (sync_u[j]) {
#pragma unroll
          for (int t = 0; t < V; ++t) {
            if (m == 0) u0[j][t] = uv[j][t];
            else mean_add(du[j][t], uv[j][t], u0[j][t]);
          }
        } else {
          store_v<float, V, NTS>(p.u[j], r, uv[j]);
        }
      }
      if constexpr (FORM != kSgdm) {
        if (sync_v) {
#pragma unroll
          for (int t = 0; t < V; ++t) {
            if (m == 0) v0[t] = vv[t];
            else mean_add(dv[t], vv[t], v0[t]);
          }
        } else {
          store_v<float, V, NTS>(p.v, r, vv);
        }
      }
    }
    // the means, written to every replica row
    if (sync_x) {
#pragma unroll
      for (int t = 0; t < V; ++t) x0[t] = mean_of(x0[t], dx[t], rk);
      outer_step<V>(p.outer, e, x0);
      for (int32_t m = 0; m < K; ++m) store_v<XT, V, NTS>(x, (int64_t)m * p.P + e, x0);
    }
#pragma unroll
    for (int j = 0; j < N; ++j) {
      if (!sync_u[j]) continue;
#pragma unroll
      for (int t = 0; t < V; ++t) u0[j][t] = mean_of(u0[j][t], du[j][t], rk);
      for (int32_t m = 0; m < K; ++m) store_v<float, V, NTS>(p.u[j], (int64_t)m * p.P + e, u0[j]);
    }
    if constexpr (FORM != kSgdm) {
      if (sync_v) {
#pragma unroll
        for (int t = 0; t < V; ++t) v0[t] = mean_of(v0[t], dv[t], rk);
        for (int32_t m = 0; m < K; ++m) store_v<float, V, NTS>(p.v, (int64_t)m * p.P + e, v0);
      }
    }
  }
}

// The same fused step + mean with one wavefront per replica (blockDim =
// 64 K, 1 < K <= kWaveMaxK): lane l of wave m updates elements
// [e, e + V) of replica m, e = tile 64 V + l V, exactly like the plain step,
// so every replica keeps its own loads in flight.  For each due state the
// updated values pass through LDS; the mean of column t of the tile is
// formed by wave t mod K as S^0 + (sum_{m>=1}(S^m - S^0)) / K in replica
// order (the arithmetic of k_replica_mean, bit for bit), the OuterOpt is
// applied to x element by element, and every wave stores the mean to its
// row.  Barriers are reached by all threads, also in the row tail.  The
// register budget is held to 8 waves per SIMD, so two 16-wave workgroups
// share a CU and one's mean phase overlaps the other's streaming.
constexpr int kWaveMaxK = 16;

template <int FORM, int N, typename XT, typename GT, int V, int NTM, int ORDER>
__global__ __launch_bounds__(64 * kWaveMaxK) __attribute__((amdgpu_waves_per_eu(8)))
void k_local_step_sync_waves(StepParams p0, uint32_t mask, int32_t K) {
  constexpr bool NTL = (NTM & 1) != 0, NTS = (NTM & 2) != 0;
  // The device-side update number's scalars take a few dozen fp64
  // operations.  Formed after a tile's loads are issued, their latency is
  // hidden, but their temporaries meet the loaded values: with six or more
  // streams loaded that exceeded the 64-register budget and spilled, so
  // those forms take them once per workgroup before any load.
  constexpr bool kEarly = 2 + N + (FORM != kSgdm ? 1 : 0) >= 6;
  const StepParams early = kEarly ? device_scalars(p0) : p0;
  constexpr int NS = 2 + N;  // x, u^1..u^N, v
  __shared__ float lds[kWaveMaxK][64 * V];
  const int32_t m = threadIdx.x >> 6, lane = threadIdx.x & 63;
  XT* __restrict__ x = reinterpret_cast<XT*>(p0.x);
  const GT* __restrict__ g = reinterpret_cast<const GT*>(p0.g);
  const double rk = 1.0 / (double)K;
  // m is the same in every lane of a wave: readfirstlane makes that visible
  const float sc =
      (FORM != kAdopt && p0.scale != nullptr) ? load_uniform(p0.scale + __builtin_amdgcn_readfirstlane(m)) : 1.0f;

  for (int64_t tile = blockIdx.x; tile < p0.tiles; tile += gridDim.x) {
    const int64_t e = tile * (int64_t)(64 * V) + (int64_t)lane * V;
    const bool in = e < p0.P;
    const int64_t r = (int64_t)m * p0.P + e;
    float val[NS][V];  // updated x, u^j, v of this lane's elements
    if (in) {
      float gv[V], uv[N][V];
      load_v<GT, V, NTL>(g, r, gv);
      load_v<XT, V, NTL>(x, r, val[0]);
#pragma unroll
      for (int j = 0; j < N; ++j) load_v<float, V, NTL>(p0.u[j], r, uv[j]);
      if constexpr (FORM != kSgdm) load_v<float, V, NTL>(p0.v, r, val[NS - 1]);
      // the step-dependent scalars after the loads are in flight
      const StepParams p = kEarly ? early : device_scalars(p0);
#pragma unroll
      for (int t = 0; t < V; ++t) {
        float uu[N];
#pragma unroll
        for (int j = 0; j < N; ++j) uu[j] = uv[j][t];
        float vt = (FORM != kSgdm) ? val[NS - 1][t] : 0.0f;
        update_element<FORM, N, ORDER>(p, sc, gv[t], val[0][t], uu, vt);
        val[0][t] = as_stored<XT>(val[0][t]);
#pragma unroll
        for (int j = 0; j < N; ++j) val[1 + j][t] = uu[j];
        val[NS - 1][t] = vt;
      }
    }
#pragma unroll
    for (int k = 0; k < NS; ++k) {
      if (FORM == kSgdm && k == NS - 1) continue;
      const bool due = ((mask >> k) & 1u) != 0;
      if (!due) {
        if (!in) continue;
        if (k == 0) store_v<XT, V, NTS>(x, r, val[0]);
        else if (k == NS - 1) store_v<float, V, NTS>(p0.v, r, val[k]);
        else store_v<float, V, NTS>(p0.u[k - 1], r, val[k]);
        continue;
      }
#pragma unroll
      for (int t = 0; t < V; ++t) lds[m][t * 64 + lane] = val[k][t];
      __syncthreads();
      // column t (element e + t of every lane) is averaged by wave t mod K
      for (int t = m; in && t < V; t += K) {
        const float s0 = lds[0][t * 64 + lane];
        double d = 0.0;
#pragma unroll 4
        for (int32_t q = 1; q < K; ++q) mean_add(d, lds[q][t * 64 + lane], s0);
        lds[0][t * 64 + lane] = mean_of(s0, d, rk);
      }
      __syncthreads();
      if (k == 0 && p0.outer.xo != nullptr) {
        outer_step_piece<V>(p0.outer, tile * (int64_t)(64 * V), p0.P, K, m, lane, &lds[0][0]);
        __syncthreads();
      }
      if (in) {
        float mean[V];
#pragma unroll
        for (int t = 0; t < V; ++t) mean[t] = lds[0][t * 64 + lane];
        if (k == 0) store_v<XT, V, NTS>(x, r, mean);
        else if (k == NS - 1) store_v<float, V, NTS>(p0.v, r, mean);
        else store_v<float, V, NTS>(p0.u[k - 1], r, mean);
      }
      __syncthreads();
    }
  }
}

// Probabilistic SGDM variant (Algorithm 4): the first moments due in mask
// are averaged over the replicas BEFORE the update direction uses them, so
// every replica steps with the averaged momentum; x is updated and, when
// bit 0 is set, averaged as in k_local_step_sync.  Two passes per column:
// pass 1 updates every replica's moments and stores the ones not due (the
// same thread reloads them in pass 2) and the means of the due ones; pass 2
// forms each replica's direction and updates x.
template <int N, typename XT, typename GT, int V, int NTM, int C = 0>
__global__ __launch_bounds__(kBlock) void k_sgdm_averaged_momenta(StepParams p0, uint32_t mask, int32_t K) {
#pragma clang fp contract(off)
  const StepParams p = device_scalars(p0);
  constexpr bool NTL = (NTM & 1) != 0, NTS = (NTM & 2) != 0;
  const bool sync_x = (mask & 1u) != 0;
  bool sync_u[N];
#pragma unroll
  for (int j = 0; j < N; ++j) sync_u[j] = ((mask >> (j + 1)) & 1u) != 0;
  XT* __restrict__ x = reinterpret_cast<XT*>(p.x);
  const GT* __restrict__ g = reinterpret_cast<const GT*>(p.g);
  const double rk = 1.0 / (double)K;

  for (int64_t tile = blockIdx.x; tile < p.tiles; tile += gridDim.x) {
    const int64_t e = tile_elem<kBlock * V, C>(tile, (int)threadIdx.x * V);
    if (e >= p.P) continue;
    // pass 1: u^j of every replica; due ones become their replica mean
    float u0[N][V];
    double du[N][V];
#pragma unroll
    for (int j = 0; j < N; ++j)
#pragma unroll
      for (int t = 0; t < V; ++t) du[j][t] = 0.0;
    for (int32_t m = 0; m < K; ++m) {
      const int64_t r = (int64_t)m * p.P + e;
      float gv[V], uv[N][V];
      load_v<GT, V, NTL>(g, r, gv);
#pragma unroll
      for (int j = 0; j < N; ++j) load_v<float, V, NTL>(p.u[j], r, uv[j]);
      const float sc = p.scale != nullptr ? load_uniform(p.scale + m) : 1.0f;
#pragma unroll
      for (int t = 0; t < V; ++t) {
        const float gh = sc * gv[t];
#pragma unroll
        for (int j = 0; j < N; ++j) uv[j][t] = __builtin_fmaf(p.beta[j], uv[j][t], p.omb[j] * gh);
      }
#pragma unroll
      for (int j = 0; j < N; ++j) {
        if (sync_u[j]) {
#pragma unroll
          for (int t = 0; t < V; ++t) {
            if (m == 0) u0[j][t] = uv[j][t];
            else mean_add(du[j][t], uv[j][t], u0[j][t]);
          }
        } else {
          store_v<float, V, false>(p.u[j], r, uv[j]);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < N; ++j) {
      if (!sync_u[j]) continue;
#pragma unroll
      for (int t = 0; t < V; ++t) u0[j][t] = mean_of(u0[j][t], du[j][t], rk);
      for (int32_t m = 0; m < K; ++m) store_v<float, V, NTS>(p.u[j], (int64_t)m * p.P + e, u0[j]);
    }
    // pass 2: direction with the averaged (due) or local (not due) moments
    float x0[V];
    double dx[V];
#pragma unroll
    for (int t = 0; t < V; ++t) dx[t] = 0.0;
    for (int32_t m = 0; m < K; ++m) {
      const int64_t r = (int64_t)m * p.P + e;
      float gv[V], xv[V], uv[N][V];
      load_v<GT, V, NTL>(g, r, gv);
      load_v<XT, V, NTL>(x, r, xv);
#pragma unroll
      for (int j = 0; j < N; ++j) {
        if (sync_u[j]) {
#pragma unroll
          for (int t = 0; t < V; ++t) uv[j][t] = u0[j][t];
        } else {
          load_v<float, V, false>(p.u[j], r, uv[j]);
        }
      }
      const float sc = p.scale != nullptr ? load_uniform(p.scale + m) : 1.0f;
#pragma unroll
      for (int t = 0; t < V; ++t) {
        const float gh = sc * gv[t];
        float delta = p.gw * gh;
#pragma unroll
        for (int j = 0; j < N; ++j) delta = __builtin_fmaf(p.w[j], uv[j][t], delta);
        xv[t] = as_stored<XT>(__builtin_fmaf(-p.lr, delta, xv[t]));
      }
      if (sync_x) {
#pragma unroll
        for (int t = 0; t < V; ++t) {
          if (m == 0) x0[t] = xv[t];
          else mean_add(dx[t], xv[t], x0[t]);
        }
      } else {
        store_v<XT, V, NTS>(x, r, xv);
      }
    }
    if (sync_x) {
#pragma unroll
      for (int t = 0; t < V; ++t) x0[t] = mean_of(x0[t], dx[t], rk);
      for (int32_t m = 0; m < K; ++m) store_v<XT, V, NTS>(x, (int64_t)m * p.P + e, x0);
    }
  }
}

// The same step with one wavefront per replica (blockDim = 64 K,
// 1 < K <= kWaveMaxK), in one pass: wave m loads g, x and every u^j of
// replica m once, updates its moments, and each due moment meets its
// replicas' values in LDS, where column t is averaged by wave t mod K (the
// mean_add / mean_of order of every averaging kernel) and read back by
// every wave before the direction uses it; x is updated and, when due,
// averaged the same way.  The values equal k_sgdm_averaged_momenta's bit
// for bit; that kernel re-reads g (and the moments not due) in its second
// pass.  Barriers are reached by every thread, also in the row tail.
template <int N, typename XT, typename GT, int V, int NTM>
__global__ __launch_bounds__(64 * kWaveMaxK) __attribute__((amdgpu_waves_per_eu(8)))
void k_sgdm_averaged_momenta_waves(StepParams p0, uint32_t mask, int32_t K) {
#pragma clang fp contract(off)
  const StepParams p = device_scalars(p0);
  constexpr bool NTL = (NTM & 1) != 0, NTS = (NTM & 2) != 0;
  __shared__ float lds[kWaveMaxK][64 * V];
  const int32_t m = threadIdx.x >> 6, lane = threadIdx.x & 63;
  XT* __restrict__ x = reinterpret_cast<XT*>(p.x);
  const GT* __restrict__ g = reinterpret_cast<const GT*>(p.g);
  const double rk = 1.0 / (double)K;
  const float sc = p.scale != nullptr ? load_uniform(p.scale + __builtin_amdgcn_readfirstlane(m)) : 1.0f;

  // the mean over the replicas of val (this wave's row values), through
  // LDS, written back into val
  auto average = [&](float (&val)[V], bool in) {
#pragma unroll
    for (int t = 0; t < V; ++t) lds[m][t * 64 + lane] = val[t];
    __syncthreads();
    for (int t = m; in && t < V; t += K) {
      const float s0 = lds[0][t * 64 + lane];
      double d = 0.0;
#pragma unroll 4
      for (int32_t q = 1; q < K; ++q) mean_add(d, lds[q][t * 64 + lane], s0);
      lds[0][t * 64 + lane] = mean_of(s0, d, rk);
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < V; ++t) val[t] = lds[0][t * 64 + lane];
    __syncthreads();
  };

  for (int64_t tile = blockIdx.x; tile < p.tiles; tile += gridDim.x) {
    const int64_t e = tile * (int64_t)(64 * V) + (int64_t)lane * V;
    const bool in = e < p.P;
    const int64_t r = (int64_t)m * p.P + e;
    float gv[V], xv[V], uv[N][V];
#pragma unroll
    for (int t = 0; t < V; ++t) gv[t] = xv[t] = 0.0f;
#pragma unroll
    for (int j = 0; j < N; ++j)
#pragma unroll
      for (int t = 0; t < V; ++t) uv[j][t] = 0.0f;
    if (in) {
      load_v<GT, V, NTL>(g, r, gv);
      load_v<XT, V, NTL>(x, r, xv);
#pragma unroll
      for (int j = 0; j < N; ++j) load_v<float, V, NTL>(p.u[j], r, uv[j]);
    }
#pragma unroll
    for (int t = 0; t < V; ++t) {
      const float gh = sc * gv[t];
#pragma unroll
      for (int j = 0; j < N; ++j) uv[j][t] = __builtin_fmaf(p.beta[j], uv[j][t], p.omb[j] * gh);
    }
#pragma unroll
    for (int j = 0; j < N; ++j) {
      if ((mask >> (j + 1)) & 1u) average(uv[j], in);
      if (in) store_v<float, V, NTS>(p.u[j], r, uv[j]);
    }
#pragma unroll
    for (int t = 0; t < V; ++t) {
      const float gh = sc * gv[t];
      float delta = p.gw * gh;
#pragma unroll
      for (int j = 0; j < N; ++j) delta = __builtin_fmaf(p.w[j], uv[j][t], delta);
      xv[t] = as_stored<XT>(__builtin_fmaf(-p.lr, delta, xv[t]));
    }
    if (mask & 1u) average(xv, in);
    if (in) store_v<XT, V, NTS>(x, r, xv);
  }
}

// ADOPT's first update with the previous-v order: v = g^2, nothing else.
template <typename GT, int V, int U, bool NT>
__global__ __launch_bounds__(kBlock) void k_adopt_init_v(const void* gp, float* vp, int64_t P, int64_t tiles) {
  const int64_t row = (int64_t)blockIdx.y * P;
  const GT* __restrict__ g = reinterpret_cast<const GT*>(gp) + row;
  float* __restrict__ v = vp + row;
  for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    const int64_t base = tile * (int64_t)(kBlock * V * U);
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t e = base + ((int64_t)k * kBlock + threadIdx.x) * V;
      if (e >= P) continue;
      float a[V];
      load_v<GT, V, NT>(g, e, a);
#pragma unroll
      for (int t = 0; t < V; ++t) a[t] = a[t] * a[t];
      store_v<float, V, NT>(v, e, a);
    }
  }
}

// --------------------------------------------------------- replica mean

struct MeanParams {
  void* state[kMaxMeanStates];  // [K][P] buffers of one storage type
  int64_t P;
  int64_t tiles;
  int32_t K;
  int32_t outer_state;          // index of x in state[] when OuterOpt applies, else -1
  OuterParams outer;
};

// E_m[S] for the state blockIdx.y: every element becomes
// S^0 + (sum_{m>=1} (S^m - S^0)) / K (mean_of) and is stored to all K rows.
// Each thread reads the K rows of its own columns and writes them back, so
// the in-place update has no cross-thread hazard.
template <typename T, int V, bool NT, int U = 1, int C = 0>
__global__ __launch_bounds__(kBlock) void k_replica_mean(MeanParams p) {
  T* __restrict__ s = reinterpret_cast<T*>(p.state[blockIdx.y]);
  const double rk = 1.0 / (double)p.K;
  for (int64_t tile = blockIdx.x; tile < p.tiles; tile += gridDim.x) {
    float s0[U][V];
    double d[U][V];
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t e = tile_elem<kBlock * V * U, C>(tile, (k * kBlock + (int)threadIdx.x) * V);
      if (e < p.P) load_v<T, V, NT>(s, e, s0[k]);
#pragma unroll
      for (int t = 0; t < V; ++t) d[k][t] = 0.0;
    }
#pragma unroll 4
    for (int32_t m = 1; m < p.K; ++m) {
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int64_t e = tile_elem<kBlock * V * U, C>(tile, (k * kBlock + (int)threadIdx.x) * V);
        if (e >= p.P) continue;
        float a[V];
        load_v<T, V, NT>(s + (int64_t)m * p.P, e, a);
#pragma unroll
        for (int t = 0; t < V; ++t) mean_add(d[k][t], a[t], s0[k][t]);
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t e = tile_elem<kBlock * V * U, C>(tile, (k * kBlock + (int)threadIdx.x) * V);
      if (e >= p.P) continue;
#pragma unroll
      for (int t = 0; t < V; ++t) s0[k][t] = mean_of(s0[k][t], d[k][t], rk);
      if ((int32_t)blockIdx.y == p.outer_state) outer_step<V>(p.outer, e, s0[k]);
#pragma unroll 4
      for (int32_t m = 0; m < p.K; ++m) store_v<T, V, NT>(s + (int64_t)m * p.P, e, s0[k]);
    }
  }
}

// The same mean with whole waves per replica row (blockDim = 64 K / R,
// 1 < K <= kWaveMaxK, R | K; dynamic LDS of K * 64 * V floats): each
// workgroup takes one piece of 64 V consecutive elements (a 1 KiB access
// for fp32 and bf16 rows), wave w loads the pieces of rows w, w + W, ...,
// w + (R - 1) W (W = K / R waves), the K pieces meet in LDS, column t of
// the piece is averaged by wave t mod W with mean_add / mean_of in replica
// order (so every element gets exactly the value k_replica_mean gives),
// the OuterOpt runs element by element on x, and each wave stores the mean
// to its rows.  Each wave then issues R loads and R stores per piece, as a
// plain copy does; a thread that walks all K rows of its columns
// (k_replica_mean) ran the K = 4 mean at 74% of the HBM peak on MI355X,
// this kernel at 82.6%.  With K = 16 and one row per wave only two
// 16-wave workgroups fit on a CU and every barrier idles 16 waves; two rows
// per wave took the K = 16 mean from 8.2 to 7.6 ms (69% to 74.5%) and the
// K = 8 bf16 mean from 0.745 to 0.685 ms, four rows per wave gave nothing.
// Barriers are reached by every thread, also in the row tail.
template <typename T, int V, bool NT, int R = 1>
__global__ __launch_bounds__(64 * kWaveMaxK / R) void k_replica_mean_waves(MeanParams p) {
  extern __shared__ float lds_mean[];  // [K][64 V]
  T* __restrict__ s = reinterpret_cast<T*>(p.state[blockIdx.y]);
  const int32_t K = p.K, W = K / R, w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const double rk = 1.0 / (double)K;
  const bool outer = (int32_t)blockIdx.y == p.outer_state;
  for (int64_t tile = blockIdx.x; tile < p.tiles; tile += gridDim.x) {
    const int64_t e = tile * (int64_t)(64 * V) + (int64_t)lane * V;
    const bool in = e < p.P;
    float a[R][V];
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int t = 0; t < V; ++t) a[r][t] = 0.0f;
    if (in) {
#pragma unroll
      for (int r = 0; r < R; ++r) load_v<T, V, NT>(s + (int64_t)(w + r * W) * p.P, e, a[r]);
    }
#pragma unroll
    for (int r = 0; r < R; ++r)
#pragma unroll
      for (int t = 0; t < V; ++t) lds_mean[((w + r * W) * V + t) * 64 + lane] = a[r][t];
    __syncthreads();
    for (int t = w; in && t < V; t += W) {
      const float s0 = lds_mean[t * 64 + lane];
      double d = 0.0;
      for (int32_t q = 1; q < K; ++q) mean_add(d, lds_mean[(q * V + t) * 64 + lane], s0);
      lds_mean[t * 64 + lane] = mean_of(s0, d, rk);
    }
    __syncthreads();
    if (outer) {
      outer_step_piece<V>(p.outer, tile * (int64_t)(64 * V), p.P, W, w, lane, lds_mean);
      __syncthreads();
    }
    if (in) {
      float b[V];
#pragma unroll
      for (int t = 0; t < V; ++t) b[t] = lds_mean[t * 64 + lane];
#pragma unroll
      for (int r = 0; r < R; ++r) store_v<T, V, NT>(s + (int64_t)(w + r * W) * p.P, e, b);
    }
    __syncthreads();
  }
}

// ----------------------------------------------------- global-norm clip

// One 64-lane DPP move of a double (both halves), rows outside RowMask and
// lanes without a source read 0.
template <int Ctrl, int RowMask>
__device__ __forceinline__ double dpp_f64(double v) {
  const unsigned long long b = __builtin_bit_cast(unsigned long long, v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(unsigned)b, Ctrl, RowMask, 0xf, true);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(unsigned)(b >> 32), Ctrl, RowMask, 0xf, true);
  return __builtin_bit_cast(double, ((unsigned long long)(unsigned)hi << 32) | (unsigned)lo);
}

// Sum of a double over the 64 lanes of a wave, in a fixed order, returned
// as a wave-uniform value.  Quad permutes [1,0,3,2] and [2,3,0,1], the
// half-row mirror and the row mirror leave every lane with its 16-lane
// row's sum; the row-15 broadcast (rows 1 and 3) and the row-31 broadcast
// (rows 2 and 3) carry the lower rows' sums into row 3, and lane 63 holds
// the total.  DPP moves stay in the vector ALU: the xor-shuffle butterfly
// goes through ds_bpermute, two LDS permutes of 256 B per step for a
// double, and in the diagnostics kernel, which ends every workgroup with
// five such sums per wave, that LDS traffic cost more time than the
// workgroup's own data exchange.
__device__ __forceinline__ double wave_sum(double a) {
  a += dpp_f64<0xB1, 0xf>(a);   // quad_perm [1,0,3,2]
  a += dpp_f64<0x4E, 0xf>(a);   // quad_perm [2,3,0,1]
  a += dpp_f64<0x141, 0xf>(a);  // row_half_mirror
  a += dpp_f64<0x140, 0xf>(a);  // row_mirror
  a += dpp_f64<0x142, 0xa>(a);  // row_bcast:15 into rows 1, 3
  a += dpp_f64<0x143, 0xc>(a);  // row_bcast:31 into rows 2, 3
  const unsigned long long b = __builtin_bit_cast(unsigned long long, a);
  const unsigned lo = __builtin_amdgcn_readlane((int)(unsigned)b, 63);
  const unsigned hi = __builtin_amdgcn_readlane((int)(unsigned)(b >> 32), 63);
  return __builtin_bit_cast(double, ((unsigned long long)hi << 32) | lo);
}

// Partial sums of g^2 in fp64 for replica blockIdx.y; each block writes
// one partial (fixed order: deterministic for a fixed grid).
template <typename GT, int V, int U, int C = 0>
__global__ __launch_bounds__(kBlock) void k_sumsq_partial(const void* gp, int64_t P, int64_t tiles,
                                                          double* __restrict__ partials) {
  const int64_t row = (int64_t)blockIdx.y * P;
  const GT* __restrict__ g = reinterpret_cast<const GT*>(gp) + row;
  double acc = 0.0;
  for (int64_t tile = blockIdx.x; tile < tiles; tile += gridDim.x) {
    float a[U][V];
    // The thread's last slot lies furthest along the row: when it is in
    // range, all U loads are issued unconditionally, back to back, so U
    // vector loads per lane are in flight (a guarded load per slot is
    // waited on before the next is issued).
    if (tile_elem<kBlock * V * U, C>(tile, ((U - 1) * kBlock + (int)threadIdx.x) * V) < P) {
#pragma unroll
      for (int k = 0; k < U; ++k)
        load_v<GT, V, false>(g, tile_elem<kBlock * V * U, C>(tile, (k * kBlock + (int)threadIdx.x) * V), a[k]);
    } else {
#pragma unroll
      for (int k = 0; k < U; ++k) {
        const int64_t e = tile_elem<kBlock * V * U, C>(tile, (k * kBlock + (int)threadIdx.x) * V);
        if (e < P) load_v<GT, V, false>(g, e, a[k]);
      }
    }
#pragma unroll
    for (int k = 0; k < U; ++k) {
      const int64_t e = tile_elem<kBlock * V * U, C>(tile, (k * kBlock + (int)threadIdx.x) * V);
      if (e >= P) continue;
#pragma unroll
      for (int t = 0; t < V; ++t) {
        const double d = (double)a[k][t];
        acc = __builtin_fma(d, d, acc);
      }
    }
  }
  acc = wave_sum(acc);
  __shared__ double ws[kBlock / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) ws[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
#pragma unroll
    for (int i = 0; i < kBlock / 64; ++i) t += ws[i];
    partials[(int64_t)blockIdx.y * gridDim.x + blockIdx.x] = t;
  }
}

// scale[m] = min(1, rho / ||g^m||), 1 for a zero norm; one workgroup of
// kFinalizeBlock threads per replica sums that replica's nb partials in a
// fixed order (thread-strided, four independent accumulators per thread so
// four loads are in flight, then waves in order): deterministic for a given
// nb, and short next to the norm pass even with one partial per 4096
// elements.
constexpr int kFinalizeBlock = 1024;

__global__ __launch_bounds__(kFinalizeBlock) void k_clip_finalize(const double* __restrict__ partials, int32_t nb,
                                                                  double rho, float* __restrict__ scale) {
  const int32_t m = blockIdx.x;
  const double* __restrict__ q = partials + (int64_t)m * nb;
  double a0 = 0.0, a1 = 0.0, a2 = 0.0, a3 = 0.0;
  int32_t i = threadIdx.x;
  for (; i + 3 * kFinalizeBlock < nb; i += 4 * kFinalizeBlock) {
    a0 += q[i];
    a1 += q[i + kFinalizeBlock];
    a2 += q[i + 2 * kFinalizeBlock];
    a3 += q[i + 3 * kFinalizeBlock];
  }
  for (; i < nb; i += kFinalizeBlock) a0 += q[i];
  double acc = wave_sum((a0 + a1) + (a2 + a3));
  __shared__ double ws[kFinalizeBlock / 64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  if (lane == 0) ws[wave] = acc;
  __syncthreads();
  if (threadIdx.x == 0) {
    double t = 0.0;
#pragma unroll
    for (int w = 0; w < kFinalizeBlock / 64; ++w) t += ws[w];
    const double norm = __builtin_sqrt(t);
    double c = 1.0;
    if (norm > 0.0) {
      c = rho / norm;
      if (!(c < 1.0)) c = 1.0;
    }
    scale[m] = (float)c;
  }
}

// ------------------------------------------------ averaging diagnostics

constexpr int kStatsMaxK = 16;
constexpr int kStatsStride = 4 + 2 * kStatsMaxK;  // doubles per state (layout in mtdao.h)

// The replica mean of the wave-per-replica kernel (same pieces, same
// mean_add / mean_of order, same values) plus, from the values before
// averaging, the averaging diagnostics of state blockIdx.y: ||cbar||^2,
// sum_m ||c^m - cbar||^2, ||xo||^2, ||c^m||^2 and <c^m, cbar>, with
// c^m = S^m, or c^m = xo - x^m for x under a Nesterov OuterOpt.
// blockDim = 64 K (1 <= K <= kStatsMaxK), dynamic LDS of K * 64 * V
// floats.  Workgroup b takes q pieces of 64 V elements, pieces
// ((b / 8) q + i) 8 + b mod 8 for i < q: each XCD keeps one piece in eight,
// and as workgroups are dispatched in order the pieces in flight stay a
// compact window, as in the plain mean (a fixed grid of workgroups
// striding over the row scattered them and ran 30% slower).  Each wave
// keeps fp64 sums for its own replica (wave 0 also those of cbar and xo):
// a lane forms the V products of a piece in fp32 (one rounding each, about
// 6e-8 relative) and adds their fp32 sum to the fp64 sums, which keeps the
// fp64 work per element to a fraction of an operation.  The workgroup
// writes its kStatsSums(K) sums, contiguous, to
// partials[state][workgroup][sum]:
//   0 ||cbar||^2, 1 sum_m ||c^m - cbar||^2, 2 ||xo||^2,
//   3 + m ||c^m||^2, 3 + K + m <c^m, cbar>.
__host__ __device__ constexpr int kStatsSums(int K) { return 3 + 2 * K; }

template <typename T, int V>
__global__ __launch_bounds__(64 * kStatsMaxK) void k_replica_mean_stats(MeanParams p, int32_t q,
                                                                          double* __restrict__ partials) {
  extern __shared__ float lds_stats[];  // [K][64 V]
  __shared__ double red[kStatsMaxK][5];
  T* __restrict__ s = reinterpret_cast<T*>(p.state[blockIdx.y]);
  const int32_t K = p.K, m = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const bool outer = (int32_t)blockIdx.y == p.outer_state && p.outer.xo != nullptr;
  const double rk = 1.0 / (double)K;
  T* __restrict__ row = s + (int64_t)m * p.P;
  double a_sq = 0.0, a_dot = 0.0, a_var = 0.0, a_mean = 0.0, a_ref = 0.0;
  for (int32_t i = 0; i < q; ++i) {
    const int64_t tile = ((int64_t)(blockIdx.x >> 3) * q + i) * 8 + (blockIdx.x & 7);
    if (tile >= p.tiles) break;  // uniform over the workgroup
    const int64_t e = tile * (int64_t)(64 * V) + (int64_t)lane * V;
    const bool in = e < p.P;
    float a[V], xo[V];
#pragma unroll
    for (int t = 0; t < V; ++t) a[t] = xo[t] = 0.0f;
    if (in) {
      load_v<T, V, true>(row, e, a);
      if (outer) load_v<float, V, false>(p.outer.xo, e, xo);
    }
#pragma unroll
    for (int t = 0; t < V; ++t) lds_stats[(m * V + t) * 64 + lane] = a[t];
    __syncthreads();
    for (int t = m; in && t < V; t += K) {
      const float s0 = lds_stats[t * 64 + lane];
      double d = 0.0;
      for (int32_t q = 1; q < K; ++q) mean_add(d, lds_stats[(q * V + t) * 64 + lane], s0);
      lds_stats[t * 64 + lane] = mean_of(s0, d, rk);
    }
    __syncthreads();
    float mean[V];
#pragma unroll
    for (int t = 0; t < V; ++t) mean[t] = lds_stats[t * 64 + lane];
    if (outer) {
      __syncthreads();  // every wave has read the means before the outer step rewrites them
      outer_step_piece<V>(p.outer, tile * (int64_t)(64 * V), p.P, K, m, lane, lds_stats);
      __syncthreads();
    }
    // store first, then reduce the diagnostics while the stores drain
    if (in) {
      float out[V];
#pragma unroll
      for (int t = 0; t < V; ++t) out[t] = outer ? lds_stats[t * 64 + lane] : mean[t];
      store_v<T, V, true>(row, e, out);
      // the piece's V terms in fp32, added to the fp64 sums once per piece
      float f_sq = 0.0f, f_dot = 0.0f, f_var = 0.0f, f_mean = 0.0f, f_ref = 0.0f;
#pragma unroll
      for (int t = 0; t < V; ++t) {
        const float cbar = outer ? xo[t] - mean[t] : mean[t];
        const float c = outer ? xo[t] - a[t] : a[t];
        const float dv = a[t] - mean[t];  // c - cbar up to sign
        f_sq = __builtin_fmaf(c, c, f_sq);
        f_dot = __builtin_fmaf(c, cbar, f_dot);
        f_var = __builtin_fmaf(dv, dv, f_var);
        if (m == 0) {
          f_mean = __builtin_fmaf(cbar, cbar, f_mean);
          if (outer) f_ref = __builtin_fmaf(xo[t], xo[t], f_ref);
        }
      }
      a_sq += (double)f_sq;
      a_dot += (double)f_dot;
      a_var += (double)f_var;
      if (m == 0) {
        a_mean += (double)f_mean;
        if (outer) a_ref += (double)f_ref;
      }
    }
    __syncthreads();
  }
  // the workgroup's sums, fixed order
  const double sq = wave_sum(a_sq), dot = wave_sum(a_dot), var = wave_sum(a_var);
  const double mn = wave_sum(a_mean), ref = wave_sum(a_ref);
  if (lane == 0) {
    red[m][0] = sq;
    red[m][1] = dot;
    red[m][2] = var;
    red[m][3] = mn;
    red[m][4] = ref;
  }
  __syncthreads();
  const int ns = kStatsSums(K);
  if ((int)threadIdx.x < ns) {
    const int k = threadIdx.x;
    double v = 0.0;
    if (k == 0) v = red[0][3];
    else if (k == 1) for (int32_t q = 0; q < K; ++q) v += red[q][2];
    else if (k == 2) v = red[0][4];
    else if (k < 3 + K) v = red[k - 3][0];
    else v = red[k - 3 - K][1];
    partials[((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * ns + k] = v;
  }
}

// Fixed-order reduction of the workgroup sums, in two levels.  Each thread
// adds whole rows of kStatsSums(K) sums (contiguous in memory) in row
// order, keeping every sum in its own fp64 register, then the block adds
// the threads' totals wave by wave in order.
constexpr int kStatsChunk = 8192;
constexpr int kStatsMaxSums = 3 + 2 * kStatsMaxK;

__device__ __forceinline__ void stats_block_sum(double (&acc)[kStatsMaxSums], int ns, double* __restrict__ dst) {
  __shared__ double red[4][kStatsMaxSums];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
#pragma unroll
  for (int k = 0; k < kStatsMaxSums; ++k) {
    if (k < ns) {
      const double w = wave_sum(acc[k]);
      if (lane == 0) red[wave][k] = w;
    }
  }
  __syncthreads();
  if ((int)threadIdx.x < ns) {
    const int k = threadIdx.x;
    dst[k] = (red[0][k] + red[1][k]) + (red[2][k] + red[3][k]);
  }
}

// Level 1: chunk blockIdx.x (kStatsChunk consecutive workgroup rows) of
// state blockIdx.y into level1[state][chunk][sum].
__global__ __launch_bounds__(256) void k_stats_reduce(const double* __restrict__ partials, int64_t nb, int32_t ns,
                                                     double* __restrict__ level1) {
  double acc[kStatsMaxSums];
#pragma unroll
  for (int k = 0; k < kStatsMaxSums; ++k) acc[k] = 0.0;
  const double* __restrict__ q = partials + (int64_t)blockIdx.y * nb * ns;
  const int64_t lo = (int64_t)blockIdx.x * kStatsChunk;
  const int64_t hi = lo + kStatsChunk < nb ? lo + kStatsChunk : nb;
  for (int64_t b = lo + threadIdx.x; b < hi; b += 256) {
#pragma unroll
    for (int k = 0; k < kStatsMaxSums; ++k)
      if (k < ns) acc[k] += q[b * ns + k];
  }
  stats_block_sum(acc, ns, level1 + ((int64_t)blockIdx.y * gridDim.x + blockIdx.x) * ns);
}

// Level 2: the nc chunk rows of state blockIdx.x, in chunk order, into out
// in the layout of mtdao.h (kStatsStride doubles per state; slot 3 and the
// slots of workers m >= K are 0); the variance sum is divided by K.
__global__ __launch_bounds__(256) void k_stats_finalize(const double* __restrict__ level1, int32_t nc, int32_t K,
                                                       double* __restrict__ out) {
  __shared__ double tot[kStatsMaxSums];
  const int32_t state = blockIdx.x, ns = kStatsSums(K);
  double acc[kStatsMaxSums];
#pragma unroll
  for (int k = 0; k < kStatsMaxSums; ++k) acc[k] = 0.0;
  const double* __restrict__ q = level1 + (int64_t)state * nc * ns;
  for (int32_t c = threadIdx.x; c < nc; c += 256) {
#pragma unroll
    for (int k = 0; k < kStatsMaxSums; ++k)
      if (k < ns) acc[k] += q[(int64_t)c * ns + k];
  }
  stats_block_sum(acc, ns, tot);
  __syncthreads();
  if (threadIdx.x < kStatsStride) {
    const int k = threadIdx.x;
    double t = 0.0;
    if (k < 3) t = tot[k];
    else if (k >= 4 && k < 4 + K) t = tot[3 + (k - 4)];
    else if (k >= 4 + kStatsMaxK && k < 4 + kStatsMaxK + K) t = tot[3 + K + (k - 4 - kStatsMaxK)];
    out[(int64_t)state * kStatsStride + k] = (k == 1) ? t / (double)K : t;
  }
}

// ------------------------------------------------------------ init

// Rows 1..K-1 of x <- row 0 (every worker starts from the same x_0).
template <typename T>
__global__ __launch_bounds__(kBlock) void k_broadcast_row0(T* __restrict__ x, int64_t P, int32_t K) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < P; i += stride) {
    const T a = x[i];
    for (int32_t m = 1; m < K; ++m) x[(int64_t)m * P + i] = a;
  }
}

// xo[i] = x[0][i] widened to fp32 (the outer parameters start at x_0).
template <typename T>
__global__ __launch_bounds__(kBlock) void k_row0_to_f32(const T* __restrict__ x, float* __restrict__ xo, int64_t P) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < P; i += stride) {
    if constexpr (sizeof(T) == 2) xo[i] = bf16_to_f32(x[i]);
    else xo[i] = x[i];
  }
}

__global__ __launch_bounds__(kBlock) void k_fill_zero(float* __restrict__ a, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * kBlock;
  for (int64_t i = (int64_t)blockIdx.x * kBlock + threadIdx.x; i < n; i += stride) a[i] = 0.0f;
}

}  // namespace mtdao
