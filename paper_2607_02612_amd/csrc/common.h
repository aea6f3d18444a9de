// Device helpers shared by the gfx950 kernels of the library.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace fusion {

typedef uint16_t bf16_t;  // bfloat16 bit pattern

// Live-batch counters kept on the device so that no launch needs the host to
// know how many samples or token rows survived the previous block.
struct LiveCounts {
  int nlive;  // live samples
  int M;      // packed token rows of the live samples
};

// float -> bfloat16, round to nearest, ties to even.
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (bf16_t)(u >> 16);
}
__device__ __forceinline__ float bf16_to_f32(bf16_t h) {
  return __uint_as_float(((uint32_t)h) << 16);
}

// Storage-type conversion for the two precision paths: on the bf16 path the
// stored activations are rounded to bfloat16, on the fp32 path they are not.
template <typename T> struct St;
template <> struct St<float> {
  static __device__ __forceinline__ float put(float f) { return f; }
  static __device__ __forceinline__ float get(float v) { return v; }
};
template <> struct St<bf16_t> {
  static __device__ __forceinline__ bf16_t put(float f) { return f32_to_bf16(f); }
  static __device__ __forceinline__ float get(bf16_t v) { return bf16_to_f32(v); }
};

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}
__device__ __forceinline__ int wave_sum_i(int v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}

// Block-wide sum for blockDim.x == 256 (4 waves); `red` holds >= 4 floats.
__device__ __forceinline__ float block_sum256(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}
__device__ __forceinline__ float block_max256(float v, float* red) {
  v = wave_max(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  return fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
}
__device__ __forceinline__ int block_sum256_i(int v, int* red) {
  v = wave_sum_i(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// Exact GELU, 0.5 v (1 + erf(v / sqrt 2)).
__device__ __forceinline__ float gelu_erf(float v) {
  return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f));
}

}  // namespace fusion
