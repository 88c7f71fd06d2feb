// Reference streaming kernels for the benchmark (not part of the optimizer
// ABI): a plain copy, a read-only reduction and a write-only fill of float4
// vectors, and a bare stream with the local step's exact access mix.  They
// give the achievable HBM bandwidth of each access mix on the device and a
// copy of known size for calibrating the HBM byte counters.

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <string.h>

#include <type_traits>

#include "kernels.hpp"

typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

// Element i of tile t: the tile's 4 pieces of 64 float4 (1 KiB) lie 8
// pieces apart and the 8 tiles of a group interleave, so each of the 8 XCDs
// (round-robin dispatch) takes one 1 KiB piece in eight -- the placement the
// optimizer kernels use, and the fastest one measured for every access mix.
__device__ __forceinline__ int64_t piece_elem(int64_t t) {
  const int64_t j = threadIdx.x >> 6, lane = threadIdx.x & 63;
  return (((t >> 3) * 4 + j) * 8 + (t & 7)) * 64 + lane;
}

__global__ __launch_bounds__(256) void k_copy(const f32x4* __restrict__ a, f32x4* __restrict__ b, int64_t n4) {
  const int64_t i = piece_elem(blockIdx.x);
  if (i < n4) __builtin_nontemporal_store(__builtin_nontemporal_load(a + i), b + i);
}

__global__ __launch_bounds__(256) void k_read(const f32x4* __restrict__ a, float* __restrict__ sink, int64_t n4) {
  const int64_t i = piece_elem(blockIdx.x);
  if (i >= n4) return;
  const f32x4 v = __builtin_nontemporal_load(a + i);
  if ((v.x + v.y) + (v.z + v.w) == -1.0f) sink[0] = 1.0f;  // keeps the load alive; never true for the bench data
}

__global__ __launch_bounds__(256) void k_fill(f32x4* __restrict__ b, int64_t n4) {
  const int64_t i = piece_elem(blockIdx.x);
  const f32x4 z = {1.0f, 1.0f, 1.0f, 1.0f};
  if (i < n4) __builtin_nontemporal_store(z, b + i);
}

// Tiles covering n4 float4: whole groups of 8 tiles of 4 pieces (one tile
// per workgroup, so n4 is limited to 2^31 - 8 tiles of 256 float4).
constexpr int64_t kMaxN4 = (INT64_C(0x7fffffff) - 8) * 256;
unsigned blocks(int64_t n4) {
  const int64_t pieces = (n4 + 63) / 64;
  const int64_t b = (pieces + 31) / 32 * 8;
  return (unsigned)(b < 8 ? 8 : b);
}

// The local step's memory traffic without its arithmetic: the loop of
// k_local_step (same tile placement, 4-element slots, one slot per thread,
// nontemporal loads and stores, the same windows per row) reading g, x,
// u^1..u^N and v, and storing x, u^j and v back unchanged.  The store is
// kept by a comparison with `guard` (NaN: never true) that depends on every
// loaded value, so no load is dropped and the buffers keep their contents.
template <int N, bool HAS_V, typename XT, typename GT, int WIN>
__global__ __launch_bounds__(mtdao::kBlock) void k_step_mix(mtdao::StepParams p, float guard) {
  using namespace mtdao;
  constexpr int V = 4, T = kBlock * V, C = 64 * V;
  for (int64_t tile = blockIdx.x; tile < p.tiles; tile += gridDim.x) {
    const int64_t w = tile & 1, wt = tile >> 1;
    int64_t m = blockIdx.y, base = 0, end = p.P;
    if constexpr (WIN == kWinHalves) {
      base = w * p.wlen;
      end = w == 0 ? p.wlen : p.P;
    } else {
      m += w * (int64_t)gridDim.y;
      if (m >= p.replicas) continue;
    }
    const int64_t row = m * p.P;
    XT* __restrict__ x = reinterpret_cast<XT*>(p.x) + row;
    const GT* __restrict__ g = reinterpret_cast<const GT*>(p.g) + row;
    const int64_t e = base + tile_elem<T, C>(wt, (int)threadIdx.x * V);
    if (e >= end) continue;
    float gv[V], xv[V], uv[N][V], vv[V];
    load_v<GT, V, true>(g, e, gv);
    load_v<XT, V, true>(x, e, xv);
#pragma unroll
    for (int j = 0; j < N; ++j) load_v<float, V, true>(p.u[j] + row, e, uv[j]);
    if constexpr (HAS_V) load_v<float, V, true>(p.v + row, e, vv);
    float sum = 0.0f;
#pragma unroll
    for (int t = 0; t < V; ++t) {
      sum += gv[t] + xv[t];
#pragma unroll
      for (int j = 0; j < N; ++j) sum += uv[j][t];
      if constexpr (HAS_V) sum += vv[t];
    }
    if (sum == guard) xv[0] += 1.0f;
    store_v<XT, V, true>(x, e, xv);
#pragma unroll
    for (int j = 0; j < N; ++j) store_v<float, V, true>(p.u[j] + row, e, uv[j]);
    if constexpr (HAS_V) store_v<float, V, true>(p.v + row, e, vv);
  }
}

template <int N, bool HAS_V, typename XT, typename GT>
void launch_step_mix(mtdao::StepParams p, int32_t K, hipStream_t st) {
  using namespace mtdao;
  constexpr int T = kBlock * 4, C = 256;
  if (K > 1) {
    p.tiles = 2 * tiles_for<T, C>(p.P);
    hipLaunchKernelGGL((k_step_mix<N, HAS_V, XT, GT, kWinPairs>), dim3((unsigned)p.tiles, (K + 1) / 2),
                       dim3(kBlock), 0, st, p, __builtin_nanf(""));
  } else {
    p.wlen = ((p.P + 1) / 2 + T - 1) / T * T;
    if (p.wlen > p.P) p.wlen = p.P;
    p.tiles = 2 * tiles_for<T, C>(p.wlen);
    hipLaunchKernelGGL((k_step_mix<N, HAS_V, XT, GT, kWinHalves>), dim3((unsigned)p.tiles, K), dim3(kBlock), 0, st,
                       p, __builtin_nanf(""));
  }
}

}  // namespace

extern "C" {

// b[0..n4) = a[0..n4), float4 elements; a and b 16-byte aligned, disjoint.
int32_t stream_ref_copy(const void* a, void* b, int64_t n4, void* stream) {
  if (n4 < 0 || n4 > kMaxN4) return (int32_t)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_copy, dim3(blocks(n4)), dim3(256), 0, (hipStream_t)stream, (const f32x4*)a, (f32x4*)b, n4);
  return (int32_t)hipGetLastError();
}

// Reads a[0..n4); sink (one float) is written only if the data sum to -1.
int32_t stream_ref_read(const void* a, void* sink, int64_t n4, void* stream) {
  if (n4 < 0 || n4 > kMaxN4) return (int32_t)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_read, dim3(blocks(n4)), dim3(256), 0, (hipStream_t)stream, (const f32x4*)a, (float*)sink, n4);
  return (int32_t)hipGetLastError();
}

// b[0..n4) = 1.0f
int32_t stream_ref_fill(void* b, int64_t n4, void* stream) {
  if (n4 < 0 || n4 > kMaxN4) return (int32_t)hipErrorInvalidValue;
  hipLaunchKernelGGL(k_fill, dim3(blocks(n4)), dim3(256), 0, (hipStream_t)stream, (f32x4*)b, n4);
  return (int32_t)hipGetLastError();
}

// The local step's access mix over the optimizer's own [K][P] buffers:
// reads g, x, u[0..n) and v (NULL: none), writes x, u^j and v back
// unchanged.  x and g are fp32 or bf16 (x_bf16, g_bf16), the moments fp32;
// P % 4 == 0, every pointer 16-byte aligned, 1 <= n <= 4, K >= 1.
int32_t stream_ref_step_mix(void* x, const void* g, void* const* u, int32_t n, void* v, int32_t x_bf16,
                            int32_t g_bf16, int64_t P, int32_t K, void* stream) {
  using namespace mtdao;
  if (n < 1 || n > kMaxN || K < 1 || P < 4 || P % 4 != 0 || (x_bf16 != 0 && x_bf16 != 1) ||
      (g_bf16 != 0 && g_bf16 != 1) || (int64_t)K * P > (INT64_C(1) << 40))
    return (int32_t)hipErrorInvalidValue;
  StepParams p;
  memset(&p, 0, sizeof p);
  p.x = x;
  p.g = g;
  for (int j = 0; j < n; ++j) p.u[j] = reinterpret_cast<float*>(u[j]);
  p.v = reinterpret_cast<float*>(v);
  p.P = P;
  p.replicas = K;
  const hipStream_t st = (hipStream_t)stream;
  auto types = [&](auto nn, auto hv) {
    constexpr int NN = decltype(nn)::value;
    constexpr bool HV = decltype(hv)::value;
    if (!x_bf16 && !g_bf16) launch_step_mix<NN, HV, float, float>(p, K, st);
    else if (!x_bf16) launch_step_mix<NN, HV, float, uint16_t>(p, K, st);
    else if (!g_bf16) launch_step_mix<NN, HV, uint16_t, float>(p, K, st);
    else launch_step_mix<NN, HV, uint16_t, uint16_t>(p, K, st);
  };
  auto moments = [&](auto hv) {
    switch (n) {
      case 1: types(std::integral_constant<int, 1>{}, hv); break;
      case 2: types(std::integral_constant<int, 2>{}, hv); break;
      case 3: types(std::integral_constant<int, 3>{}, hv); break;
      default: types(std::integral_constant<int, 4>{}, hv); break;
    }
  };
  if (v) moments(std::true_type{});
  else moments(std::false_type{});
  return (int32_t)hipGetLastError();
}

}  // extern "C"
