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

// float -> bfloat16, round to nearest, ties to even: gfx950's
// v_cvt_pk_bf16_f32 (bit-identical to the integer formulation
// u + 0x7FFF + ((u >> 16) & 1) >> 16 on finite inputs, subnormals included).
__device__ __forceinline__ bf16_t f32_to_bf16(float f) {
  return __builtin_bit_cast(bf16_t, (__bf16)f);
}
// Two floats -> two bfloat16 (round to nearest even) in one 32-bit word,
// `lo` in the low half: a single v_cvt_pk_bf16_f32.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
  typedef float f32x2_t __attribute__((ext_vector_type(2)));
  return __builtin_bit_cast(uint32_t, __builtin_convertvector((f32x2_t){lo, hi}, bf16x2_t));
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

// Combine each lane's value with that of lane ^ 16 or lane ^ 32 through the
// gfx950 lane-swap instructions (no LDS round trip).  The swap of two copies
// of v leaves the lane's own value in one result and its partner's in the
// other; max and + are symmetric, so both lanes of a pair get the same bits.
__device__ __forceinline__ float max_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float max_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float sum_xor16(float v) {
  const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ __forceinline__ float sum_xor32(float v) {
  const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
  return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

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

// Block-wide integer sum for blockDim.x == 256 (4 waves); `red` holds >= 4 ints.
__device__ __forceinline__ int block_sum256_i(int v, int* red) {
  v = wave_sum_i(v);
  const int w = threadIdx.x >> 6, l = threadIdx.x & 63;
  __syncthreads();
  if (l == 0) red[w] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// Sum over the 32 lanes of a half wave (lanes 0-31 or 32-63) without LDS
// round trips: DPP swaps within quads (lane ^ 1, lane ^ 2), the mirrors of
// 8- and 16-lane rows, then the row swap of permlane16.  After each step the
// partners hold the same two summands in opposite order, so all 32 lanes end
// with the same bits.
template <int CTRL>
__device__ __forceinline__ float dpp_peer(float v) {
  return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float half_sum(float v) {
  v += dpp_peer<0xB1>(v);   // quad_perm [1, 0, 3, 2]
  v += dpp_peer<0x4E>(v);   // quad_perm [2, 3, 0, 1]
  v += dpp_peer<0x141>(v);  // row_half_mirror
  v += dpp_peer<0x140>(v);  // row_mirror
  return sum_xor16(v);
}

// Four floats -> storage type, one vector store.
template <typename T> struct Store4;
template <> struct Store4<float> {
  static __device__ __forceinline__ void put(float* p, float4 v) { *(float4*)p = v; }
};
template <> struct Store4<bf16_t> {
  static __device__ __forceinline__ void put(bf16_t* p, float4 v) {
    *(uint2*)p = make_uint2(pack_bf16x2(v.x, v.y), pack_bf16x2(v.z, v.w));
  }
};

// LayerNorm of one row of d fp32 values by a half wave (l = lane % 32 holds
// the 16-byte pieces l, l + 32, ...; d % 4 == 0, d <= 768): mean and biased
// variance in fp32 (two passes over the values held in registers),
// y = (x - mean) / sqrt(var + 1e-6) * g + b.  Optionally copies the row to
// `copy` on the way.
constexpr int LN_MAXV = 6;  // 16-byte pieces per lane (d <= 768)
template <typename T>
__device__ __forceinline__ void ln_row_half(const float* __restrict__ xr, int d, int l,
                                            const float* __restrict__ g,
                                            const float* __restrict__ b, T* __restrict__ out,
                                            float* __restrict__ copy) {
  const int n4 = d >> 2;
  float4 v[LN_MAXV];
  float s = 0.f;
#pragma unroll
  for (int i = 0; i < LN_MAXV; i++) {
    const int k = l + 32 * i;
    v[i] = k < n4 ? ((const float4*)xr)[k] : make_float4(0.f, 0.f, 0.f, 0.f);
    s += (v[i].x + v[i].y) + (v[i].z + v[i].w);
  }
  if (copy) {
#pragma unroll
    for (int i = 0; i < LN_MAXV; i++) {
      const int k = l + 32 * i;
      if (k < n4) ((float4*)copy)[k] = v[i];
    }
  }
  if (!out) return;
  const float mean = half_sum(s) / (float)d;
  float q = 0.f;
#pragma unroll
  for (int i = 0; i < LN_MAXV; i++) {
    const int k = l + 32 * i;
    if (k < n4) {
      const float a0 = v[i].x - mean, a1 = v[i].y - mean, a2 = v[i].z - mean, a3 = v[i].w - mean;
      q += (a0 * a0 + a1 * a1) + (a2 * a2 + a3 * a3);
    }
  }
  const float var = half_sum(q) / (float)d;
  const float rstd = 1.0f / sqrtf(var + 1e-6f);
#pragma unroll
  for (int i = 0; i < LN_MAXV; i++) {
    const int k = l + 32 * i;
    if (k < n4) {
      const float4 gg = ((const float4*)g)[k], bb = ((const float4*)b)[k];
      Store4<T>::put(out + 4 * k, make_float4(((v[i].x - mean) * rstd) * gg.x + bb.x,
                                              ((v[i].y - mean) * rstd) * gg.y + bb.y,
                                              ((v[i].z - mean) * rstd) * gg.z + bb.z,
                                              ((v[i].w - mean) * rstd) * gg.w + bb.w));
    }
  }
}

// GELU with the exact (erf) form, v Phi(v), Phi the standard normal CDF,
// written as GELU(v) = max(v, 0) - |v| Q(|v|) with the upper tail
// Q(a) = erfc(a / sqrt 2) / 2 from the rational approximation 7.1.28 of
// Abramowitz & Stegun (Handbook of Mathematical Functions):
//   erfc(z) = (1 + a1 z + a2 z^2 + a3 z^3 + a4 z^4 + a5 z^5 + a6 z^6)^-16,
//   |error| <= 3e-7,
// one reciprocal and four squarings.  z = a / sqrt 2 is folded into the
// coefficients, and the 1/2 through a common factor 2^(1/16) on all of them
// (P^-16 scales by 1/2).  The tail form has no cancellation for negative v;
// past |v| of about 11 the power underflows and the result is max(v, 0).
__device__ __forceinline__ float gelu_erf(float v) {
  const float a = fabsf(v);
  // 2^(1/16) a_k 2^(-k/2), k = 6 .. 0 (a_0 = 1)
  float p = fmaf(a, 5.621299664e-06f, 5.105520901e-05f);
  p = fmaf(a, p, 3.968613701e-05f);
  p = fmaf(a, p, 3.422739239e-03f);
  p = fmaf(a, p, 2.207699846e-02f);
  p = fmaf(a, p, 5.207516304e-02f);
  p = fmaf(a, p, 1.044273782e+00f);
  float r = __builtin_amdgcn_rcpf(p);
  r = r * r;
  r = r * r;
  r = r * r;
  r = r * r;
  // max(v, 0) as an integer maximum of the bit pattern (a negative float,
  // -0 included, is a negative integer): one instruction, where the float
  // maximum of a matrix-core result first re-canonicalises its input
  return fmaf(-a, r, __int_as_float(max(__float_as_int(v), 0)));
}

}  // namespace fusion
