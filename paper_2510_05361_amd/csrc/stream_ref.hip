// Reference streaming kernels for the benchmark (not part of the optimizer
// ABI): a plain copy, a read-only reduction and a write-only fill of float4
// vectors.  They give the achievable HBM bandwidth of each access mix on
// the device and a copy of known size for calibrating the HBM byte counters.

#include <hip/hip_runtime.h>
#include <stdint.h>

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

}  // extern "C"
