// Reference streaming kernels for the benchmark (not part of the optimizer
// ABI): a plain copy, a read-only reduction and a write-only fill of float4
// vectors.  They give the achievable HBM bandwidth of each access mix on
// the device and a copy of known size for calibrating the HBM byte counters.

#include <hip/hip_runtime.h>
#include <stdint.h>

typedef float f32x4 __attribute__((ext_vector_type(4)));

namespace {

__global__ __launch_bounds__(256) void k_copy(const f32x4* __restrict__ a, f32x4* __restrict__ b, int64_t n4) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride)
    __builtin_nontemporal_store(__builtin_nontemporal_load(a + i), b + i);
}

__global__ __launch_bounds__(256) void k_read(const f32x4* __restrict__ a, float* __restrict__ sink, int64_t n4) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  float acc = 0.0f;
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) {
    const f32x4 v = __builtin_nontemporal_load(a + i);
    acc += (v.x + v.y) + (v.z + v.w);
  }
  if (acc == -1.0f) sink[0] = acc;  // keeps the loads alive; never true for the bench data
}

__global__ __launch_bounds__(256) void k_fill(f32x4* __restrict__ b, int64_t n4) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  const f32x4 z = {1.0f, 1.0f, 1.0f, 1.0f};
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride) __builtin_nontemporal_store(z, b + i);
}

unsigned blocks(int64_t n4) {
  int64_t b = (n4 + 255) / 256;
  return (unsigned)(b < 1 ? 1 : (b > 0x7fffffff ? 0x7fffffff : b));
}

}  // namespace

extern "C" {

// b[0..n4) = a[0..n4), float4 elements; a and b 16-byte aligned, disjoint.
int32_t stream_ref_copy(const void* a, void* b, int64_t n4, void* stream) {
  hipLaunchKernelGGL(k_copy, dim3(blocks(n4)), dim3(256), 0, (hipStream_t)stream, (const f32x4*)a, (f32x4*)b, n4);
  return (int32_t)hipGetLastError();
}

// Reads a[0..n4); sink (one float) is written only if the data sum to -1.
int32_t stream_ref_read(const void* a, void* sink, int64_t n4, void* stream) {
  hipLaunchKernelGGL(k_read, dim3(blocks(n4)), dim3(256), 0, (hipStream_t)stream, (const f32x4*)a, (float*)sink, n4);
  return (int32_t)hipGetLastError();
}

// b[0..n4) = 1.0f
int32_t stream_ref_fill(void* b, int64_t n4, void* stream) {
  hipLaunchKernelGGL(k_fill, dim3(blocks(n4)), dim3(256), 0, (hipStream_t)stream, (f32x4*)b, n4);
  return (int32_t)hipGetLastError();
}

}  // extern "C"
