// Multi-head self-attention over ragged samples (Eq. 2), with proportional
// attention (scores += ln of the key token's size) and, on prune blocks, the
// per-head CLS attention row that scores tokens for pruning.
//
// Softmax uses the exact row maximum: the full score row of a query is held
// (LDS) before exponentiation.  E = exp(S - max), l = sum E in fp32, the
// stored probabilities E are rounded to the storage type before they
// multiply V, and O = (round(E) V) / l.
//
// One workgroup per (live sample, head); each of the 4 waves takes every
// 4th query row.  K and V of the (sample, head) are staged in LDS when they
// fit in 64 KB, else read from global memory.
#include "kernels.h"

namespace fusion {

template <typename T, bool STAGE>
__global__ __launch_bounds__(256) void attention_valu(AttnArgs a) {
  const int i = blockIdx.x, h = blockIdx.y;
  if (i >= a.cnt->nlive) return;
  const int base = a.cu[i], Tn = a.cu[i + 1] - base;
  if (Tn > a.T_ub) return;  // the host bound is exact; never overrun LDS
  if (h == 0 && threadIdx.x == 0 && a.token_counts)
    a.token_counts[a.live[i] * a.L + a.b0] = Tn;
  const int dh = a.dh, d = a.d, ld = 3 * d;
  const int ks = dh + (sizeof(T) == 2 ? 2 : 1);
  const T* qkv = (const T*)a.qkv;
  extern __shared__ __attribute__((aligned(16))) char smem[];
  const int Tu = a.T_ub;
  size_t off = 0;
  T* Ks = (T*)(smem + off);
  if (STAGE) off += ((size_t)Tu * ks * sizeof(T) + 15) & ~(size_t)15;
  T* Vs = (T*)(smem + off);
  if (STAGE) off += ((size_t)Tu * dh * sizeof(T) + 15) & ~(size_t)15;
  float* lnS = (float*)(smem + off);
  off += (size_t)Tu * 4;
  float* ps_all = (float*)(smem + off);
  off += (size_t)4 * Tu * 4;
  float* qs_all = (float*)(smem + off);

  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const T* kg = qkv + (size_t)base * ld + d + h * dh;
  const T* vg = qkv + (size_t)base * ld + 2 * d + h * dh;
  for (int t = threadIdx.x; t < Tn * dh; t += 256) {
    const int j = t / dh, dd = t - j * dh;
    if (STAGE) {
      Ks[j * ks + dd] = kg[(size_t)j * ld + dd];
      Vs[j * dh + dd] = vg[(size_t)j * ld + dd];
    }
  }
  for (int j = threadIdx.x; j < Tn; j += 256)
    lnS[j] = a.prop_attn ? logf(a.size[base + j]) : 0.f;
  __syncthreads();

  float* ps = ps_all + wave * Tu;
  float* qs = qs_all + wave * dh;
  T* out = (T*)a.out;
  for (int t0 = 0; t0 < Tn; t0 += 4) {
    const int t = t0 + wave;
    const bool active = t < Tn;
    float lsum = 1.f;
    if (active) {
      for (int dd = lane; dd < dh; dd += 64)
        qs[dd] = St<T>::get(qkv[(size_t)(base + t) * ld + h * dh + dd]);
    }
    __syncthreads();
    if (active) {
      float lm = -INFINITY;
      for (int j = lane; j < Tn; j += 64) {
        float dot = 0.f;
        for (int dd = 0; dd < dh; dd++) {
          const float kv = STAGE ? St<T>::get(Ks[j * ks + dd])
                                 : St<T>::get(kg[(size_t)j * ld + dd]);
          dot = fmaf(qs[dd], kv, dot);
        }
        float sj = dot * a.scale;
        if (a.prop_attn) sj = sj + lnS[j];
        ps[j] = sj;
        lm = fmaxf(lm, sj);
      }
      lm = wave_max(lm);
      float ls = 0.f;
      for (int j = lane; j < Tn; j += 64) {
        const float e = expf(ps[j] - lm);
        ps[j] = e;
        ls += e;
      }
      lsum = wave_sum(ls);
    }
    __syncthreads();
    if (active) {
      if (a.cls_scores && t == 0) {
        float* cs = a.cls_scores + ((size_t)i * a.H + h) * a.tmax;
        for (int j = lane; j < Tn; j += 64) cs[j] = ps[j] / lsum;
      }
      for (int dd = lane; dd < dh; dd += 64) {
        float acc = 0.f;
        for (int j = 0; j < Tn; j++) {
          const float p = St<T>::get(St<T>::put(ps[j]));
          const float vv = STAGE ? St<T>::get(Vs[j * dh + dd])
                                 : St<T>::get(vg[(size_t)j * ld + dd]);
          acc = fmaf(p, vv, acc);
        }
        out[(size_t)(base + t) * d + h * dh + dd] = St<T>::put(acc / lsum);
      }
    }
    __syncthreads();
  }
}

template <typename T>
hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.nlive_ub <= 0) return hipSuccess;
  const int ks = a.dh + (sizeof(T) == 2 ? 2 : 1);
  const size_t tail = (size_t)a.T_ub * 4 * 5 + (size_t)4 * a.dh * 4;
  const size_t staged = (((size_t)a.T_ub * ks * sizeof(T) + 15) & ~(size_t)15) +
                        (((size_t)a.T_ub * a.dh * sizeof(T) + 15) & ~(size_t)15) + tail;
  dim3 grid(a.nlive_ub, a.H);
  if (staged <= 65536) {
    attention_valu<T, true><<<grid, 256, staged, s>>>(a);
  } else {
    if (tail > 65536) return hipErrorInvalidValue;
    attention_valu<T, false><<<grid, 256, tail, s>>>(a);
  }
  return hipGetLastError();
}
template hipError_t launch_attention<float>(const AttnArgs&, hipStream_t);
template hipError_t launch_attention<bf16_t>(const AttnArgs&, hipStream_t);

}  // namespace fusion
