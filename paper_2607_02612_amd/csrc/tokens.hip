// Token-level kernels: run initialisation, patch extraction (Eq. 1),
// LayerNorm of packed rows (pre-norm blocks, exit and final heads), and a
// diagnostic state copy.
#include "kernels.h"

namespace fusion {

__global__ void init_kernel(float* __restrict__ x, int* __restrict__ rmap,
                            float* __restrict__ size,
                            int* __restrict__ origin, int* __restrict__ cu,
                            int* __restrict__ live, LiveCounts* cnt,
                            int* __restrict__ token_counts,
                            const float* __restrict__ cls,
                            const float* __restrict__ pos, int B, int n0,
                            int d, int L) {
  const int T0 = n0 + 1;
  const long rows = (long)B * T0;
  const long total = rows > (long)B * L ? rows : (long)B * L;
  const long cls_elems = (long)B * d;
  const long stride = (long)gridDim.x * blockDim.x;
  for (long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
       t < (total > cls_elems ? total : cls_elems); t += stride) {
    if (t < rows) {
      size[t] = 1.0f;
      origin[t] = (int)(t % T0);
      rmap[t] = (int)t;
    }
    if (t < (long)B * L) token_counts[t] = 0;
    if (t < cls_elems) {
      const int s = (int)(t / d), n = (int)(t - (long)s * d);
      x[(size_t)s * T0 * d + n] = cls[n] + pos[n];
    }
    if (t <= B) cu[t] = (int)(t * T0);
    if (t < B) live[t] = (int)t;
    if (t == 0) {
      cnt->nlive = B;
      cnt->M = (int)rows;
    }
  }
}

hipError_t launch_init(float* x, int* rmap, float* size, int* origin, int* cu, int* live,
                       LiveCounts* cnt, int* token_counts, const float* cls,
                       const float* pos, int B, int n0, int d, int L,
                       hipStream_t s) {
  long work = (long)B * (n0 + 1);
  if ((long)B * d > work) work = (long)B * d;
  if ((long)B * L > work) work = (long)B * L;
  int blocks = (int)((work + 255) / 256);
  if (blocks > 4096) blocks = 4096;
  init_kernel<<<blocks, 256, 0, s>>>(x, rmap, size, origin, cu, live, cnt,
                                     token_counts, cls, pos, B, n0, d, L);
  return hipGetLastError();
}

// images [B, C, S, S] -> patches [B*n0, C*p*p]; patch (gy, gx) in raster
// order, vector element (c, ky, kx).  One thread moves 4 consecutive pixels
// of an image row (p % 4 == 0, so they stay inside one patch): a 16-byte
// load and one vector store.  Threads walk the images in memory order, so a
// wave reads 1 KB of consecutive image bytes and every 128-byte line is
// fetched by one wave (walking the patches in output order instead split
// each line between two neighbouring patches, often handled on different
// XCDs, and read 1.67x the image bytes from HBM); the stores are runs of
// p / 4 lanes (32 bytes for p = 16) into one patch row.  Pixels past g p
// (S not a multiple of p) are skipped.  32-bit index math (the host checks
// that B * C * S * S / 4 fits).
template <typename T>
__global__ void patchify_kernel(const float* __restrict__ img, T* __restrict__ out,
                                int B, int C, int S, int p) {
  const int g = S / p, n0 = g * g, pd = C * p * p, sq = S / 4;
  const int items = B * C * S * sq;
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < items;
       t += gridDim.x * blockDim.x) {
    const int line = t / sq, x = (t - line * sq) * 4;  // line = (s C + c) S + y
    const int sc = line / S, y = line - sc * S;
    const int s = sc / C, c = sc - s * C;
    const int gy = y / p, gx = x / p;
    if (gy >= g || gx >= g) continue;
    const float4 v = *(const float4*)(img + (size_t)t * 4);
    const int row = s * n0 + gy * g + gx;
    Store4<T>::put(out + (size_t)row * pd + c * p * p + (y - gy * p) * p + (x - gx * p), v);
  }
}

template <typename T>
hipError_t launch_patchify(const float* img, T* out, int B, int C, int S,
                           int p, hipStream_t s) {
  const long items = (long)B * C * S * S / 4;
  if (items >= (1L << 31) || p % 4 != 0 || S % 4 != 0) return hipErrorInvalidValue;
  int blocks = (int)((items + 255) / 256);
  if (blocks > 16384) blocks = 16384;
  patchify_kernel<T><<<blocks, 256, 0, s>>>(img, out, B, C, S, p);
  return hipGetLastError();
}
template hipError_t launch_patchify<float>(const float*, float*, int, int, int, int, hipStream_t);
template hipError_t launch_patchify<bf16_t>(const float*, bf16_t*, int, int, int, int, hipStream_t);

// One half wave per row (8 rows per 256-thread workgroup), 16-byte loads and
// vector stores; the row arithmetic is ln_row_half.
template <typename T>
__global__ __launch_bounds__(256) void layernorm_kernel(
    const float* __restrict__ x, const int* __restrict__ rmap, const float* __restrict__ g,
    const float* __restrict__ bb, T* __restrict__ out, int d,
    const LiveCounts* cnt, const int* __restrict__ cu,
    const int* __restrict__ live, int cls_only, int* exit_block, int L) {
  const int lane = threadIdx.x & 63;
  const int row = blockIdx.x * 8 + (threadIdx.x >> 5);
  const int nrows = cls_only ? cnt->nlive : cnt->M;
  if (row >= nrows) return;
  const size_t src = (size_t)rmap[cls_only ? cu[row] : row];
  ln_row_half<T>(x + src * d, d, lane & 31, g, bb, out + (size_t)row * d, nullptr);
  if (exit_block && (lane & 31) == 0) exit_block[live[row]] = L;
}

template <typename T>
hipError_t launch_layernorm(const float* x, const int* rmap, const float* g, const float* b,
                            T* out, int d, const LiveCounts* cnt,
                            const int* cu, const int* live, int cls_only,
                            int rows_ub, int* exit_block, int L,
                            hipStream_t s) {
  if (rows_ub <= 0) return hipSuccess;
  if (d > 4 * 32 * LN_MAXV || d % 4 != 0) return hipErrorInvalidValue;
  layernorm_kernel<T><<<(rows_ub + 7) / 8, 256, 0, s>>>(
      x, rmap, g, b, out, d, cnt, cu, live, cls_only, exit_block, L);
  return hipGetLastError();
}
template hipError_t launch_layernorm<float>(const float*, const int*, const float*, const float*,
                                            float*, int,
                                            const LiveCounts*, const int*, const int*, int, int,
                                            int*, int, hipStream_t);
template hipError_t launch_layernorm<bf16_t>(const float*, const int*, const float*, const float*,
                                             bf16_t*,
                                             int, const LiveCounts*, const int*, const int*, int,
                                             int, int*, int, hipStream_t);

// SpatialPool input of a pooled exit head: per live sample i,
//   p = sum_t s_t x_t / sum_t s_t over its patch rows t = 1 .. T-1
// (zero vector when T = 1), then out[i] = LN(p) with (g, b) in the storage
// type of the precision path.  One 256-thread workgroup per sample: wave w
// sums rows 1 + w, 5 + w, ... (lane l holds the 16-byte pieces l, l + 64,
// l + 128), the four partial sums are added in wave order, and half wave 0
// normalises the pooled row.  The pool reads the state before the block's
// merge: size-weighted merging keeps sum_t s_t x_t and sum_t s_t, so the
// pooled vector is the same before and after it.
constexpr int POOL_MAXV = 3;  // 16-byte pieces per lane (d <= 768)
template <typename T>
__global__ __launch_bounds__(256) void pool_ln_kernel(
    const float* __restrict__ x, const int* __restrict__ rmap, const float* __restrict__ size,
    const int* __restrict__ cu, const LiveCounts* cnt,
    const float* __restrict__ g, const float* __restrict__ bb,
    T* __restrict__ out, int d) {
  const int i = blockIdx.x;
  if (i >= cnt->nlive) return;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int base = cu[i], Tn = cu[i + 1] - base, n4 = d >> 2;
  __shared__ __attribute__((aligned(16))) float part[4][4 * 64 * POOL_MAXV];
  __shared__ float pden[4];
  __shared__ __attribute__((aligned(16))) float pooled[4 * 64 * POOL_MAXV];
  float4 acc[POOL_MAXV];
#pragma unroll
  for (int k = 0; k < POOL_MAXV; k++) acc[k] = make_float4(0.f, 0.f, 0.f, 0.f);
  float den = 0.f;
  for (int t = 1 + wave; t < Tn; t += 4) {
    const float st = size[base + t];
    const float4* xr = (const float4*)(x + (size_t)rmap[base + t] * d);
#pragma unroll
    for (int k = 0; k < POOL_MAXV; k++) {
      const int q = lane + 64 * k;
      if (q < n4) {
        const float4 v = xr[q];
        acc[k].x = fmaf(st, v.x, acc[k].x);
        acc[k].y = fmaf(st, v.y, acc[k].y);
        acc[k].z = fmaf(st, v.z, acc[k].z);
        acc[k].w = fmaf(st, v.w, acc[k].w);
      }
    }
    den += st;
  }
#pragma unroll
  for (int k = 0; k < POOL_MAXV; k++) {
    const int q = lane + 64 * k;
    if (q < n4) *(float4*)&part[wave][4 * q] = acc[k];
  }
  if (lane == 0) pden[wave] = den;
  __syncthreads();
  const float D = ((pden[0] + pden[1]) + pden[2]) + pden[3];
  for (int f = tid; f < d; f += 256) {
    const float num = ((part[0][f] + part[1][f]) + part[2][f]) + part[3][f];
    pooled[f] = D > 0.f ? num / D : 0.f;
  }
  __syncthreads();
  if (tid < 32) ln_row_half<T>(pooled, d, tid, g, bb, out + (size_t)i * d, nullptr);
}

template <typename T>
hipError_t launch_pool_ln(const float* x, const int* rmap, const float* size, const int* cu,
                          const LiveCounts* cnt, const float* g, const float* b,
                          T* out, int d, int nlive_ub, hipStream_t s) {
  if (nlive_ub <= 0) return hipSuccess;
  if (d % 4 != 0 || d > 4 * 64 * POOL_MAXV) return hipErrorInvalidValue;
  pool_ln_kernel<T><<<nlive_ub, 256, 0, s>>>(x, rmap, size, cu, cnt, g, b, out, d);
  return hipGetLastError();
}
template hipError_t launch_pool_ln<float>(const float*, const int*, const float*, const int*,
                                          const LiveCounts*, const float*, const float*,
                                          float*, int, int, hipStream_t);
template hipError_t launch_pool_ln<bf16_t>(const float*, const int*, const float*, const int*,
                                           const LiveCounts*, const float*, const float*,
                                           bf16_t*, int, int, hipStream_t);

__global__ void step_init_kernel(int* __restrict__ live, int B, int* __restrict__ rmap, int M,
                                 LiveCounts* cnt) {
  const int n = B > M ? B : M;
  for (int t = blockIdx.x * blockDim.x + threadIdx.x; t < n; t += gridDim.x * blockDim.x) {
    if (t < B) live[t] = t;
    if (t < M) rmap[t] = t;
    if (t == 0) {
      cnt->nlive = B;
      cnt->M = M;
    }
  }
}

hipError_t launch_step_init(int* live, int B, int* rmap, int M, LiveCounts* cnt,
                            hipStream_t s) {
  const int n = B > M ? B : M;
  int blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  if (blocks < 1) blocks = 1;
  step_init_kernel<<<blocks, 256, 0, s>>>(live, B, rmap, M, cnt);
  return hipGetLastError();
}

__global__ void copy_state_kernel(const float* __restrict__ x, const int* rmap, const int* cu,
                                  const int* live, const LiveCounts* cnt,
                                  float* __restrict__ x_out, int* cu_out,
                                  int* live_out, int d) {
  const int nl = cnt->nlive;
  const long n = (long)cnt->M * d;
  for (long t = (long)blockIdx.x * blockDim.x + threadIdx.x; t < n;
       t += (long)gridDim.x * blockDim.x)
    x_out[t] = x[(size_t)rmap[t / d] * d + t % d];
  const long t = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t <= nl) cu_out[t] = cu[t];
  if (t < nl) live_out[t] = live[t];
}

hipError_t launch_copy_state(const float* x, const int* rmap, const int* cu, const int* live,
                             const LiveCounts* cnt, float* x_out, int* cu_out,
                             int* live_out, int d, int rows_ub, int nlive_ub,
                             hipStream_t s) {
  long work = (long)rows_ub * d;
  int blocks = (int)((work + 255) / 256);
  const int need = (nlive_ub + 1 + 255) / 256;
  if (blocks > 8192) blocks = 8192;
  if (blocks < need) blocks = need;
  copy_state_kernel<<<blocks, 256, 0, s>>>(x, rmap, cu, live, cnt, x_out, cu_out,
                                           live_out, d);
  return hipGetLastError();
}

}  // namespace fusion
