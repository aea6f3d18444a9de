// Multi-head self-attention over ragged samples (Eq. 2), with proportional
// attention (scores += ln of the key token's size) and, on prune blocks, the
// per-head CLS attention row that scores tokens for pruning.
//
// Softmax uses the exact row maximum: the full score row of a query is held
// (LDS or registers) before exponentiation.  E = exp(S - max), l = sum E in
// fp32, the stored probabilities E are rounded to the storage type before
// they multiply V, and O = (round(E) V) / l.  The MFMA kernels evaluate the
// exponent in base 2 with the hardware exp2: t = dot (scale log2 e) +
// ln(size) log2 e, E = exp2(t - max t) (the same quantity up to the
// rounding of the folded constants), and scale O by 1 / l.
//
// bf16 path with 64-wide heads: MFMA kernel below.  fp32 path (and any
// other head width): one workgroup per (live sample, head); each of the 4
// waves takes every 4th query row; K and V of the (sample, head) are staged
// in LDS when they fit in 64 KB, else read from global memory.
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

// ------------------------------------------------------------ bf16 MFMA --
// One workgroup per (live sample, head, block of 64 queries); each wave owns
// 16 queries.  Scores are computed transposed, S^T = K Q^T, with
// v_mfma_f32_16x16x32_bf16 so that every lane holds the scores of ONE query
// (column l%16 of the output tile) for keys 16t + 4(l/16) + j: the exact row
// maximum and the row sum are reductions over the lane's registers plus two
// xor-shuffles (lanes l, l^16, l^32, l^48 share a query).  Keys are streamed
// through LDS in chunks of 64 (K row-major; V transposed to [dh][key]), so
// any length up to 16 * MAXT keys fits.  For O = P V the lane's own
// probabilities of key tiles 2p and 2p+1 form the MFMA A operand directly:
// the 8 k-slots of lane l map to keys {32p + 4g + i, 32p + 16 + 4g + i}
// (g = l/16, i < 4), and the V operand is read from the transposed chunk
// with the same key permutation (two 8-byte reads).
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

constexpr float kLog2e = 1.4426950408889634f;
constexpr int AKC = 64;            // keys per LDS chunk
constexpr int AKS = 64 + 8;        // K chunk row stride (bf16), dh = 64
constexpr int AVS = AKC + 8;       // V^T chunk row stride (bf16)

template <int MAXT>
__global__ __launch_bounds__(256) void attention_mfma(AttnArgs a) {
  const int i = blockIdx.x, h = blockIdx.y, qb = blockIdx.z;
  if (i >= a.cnt->nlive) return;
  const int base = a.cu[i], Tn = a.cu[i + 1] - base;
  if (Tn > a.T_ub || Tn > 16 * MAXT) return;  // the host bound is exact
  if (qb * 64 >= Tn) return;
  if (h == 0 && qb == 0 && threadIdx.x == 0 && a.token_counts)
    a.token_counts[a.live[i] * a.L + a.b0] = Tn;
  const int d = a.d, ld = 3 * d;
  const float sc2 = a.scale * kLog2e;
  const bf16_t* qkv = (const bf16_t*)a.qkv;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[AKC * AKS];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[64 * AVS];
  __shared__ float lnS[16 * MAXT];

  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c = lane & 15;
  const int q0 = qb * 64 + wave * 16;   // first query of this wave
  const int nkt = (Tn + 15) >> 4;       // key tiles
  const int nch = (Tn + AKC - 1) / AKC; // key chunks

  for (int j = tid; j < nkt * 16; j += 256)
    lnS[j] = (j < Tn && a.prop_attn) ? logf(a.size[base + j]) * kLog2e : 0.f;

  // Q^T operand: lane holds Q[q0 + c][8g .. 8g+7] and [32 + 8g ..]
  bf16x8_t qop[2];
  {
    const int q = q0 + c;
    const bf16_t* qr = qkv + (size_t)(base + q) * ld + h * 64;
    for (int hf = 0; hf < 2; hf++) {
      uint4 v = make_uint4(0, 0, 0, 0);
      if (q < Tn) v = *(const uint4*)(qr + hf * 32 + 8 * g);
      qop[hf] = *(bf16x8_t*)&v;
    }
  }

  // ---- phase 1: S^T tiles for all keys
  f32x4_t S[MAXT];
#pragma unroll
  for (int t = 0; t < MAXT; t++) S[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const bf16_t* kg = qkv + (size_t)base * ld + d + h * 64;
  for (int ch = 0; ch < nch; ch++) {
    __syncthreads();
    // stage 64 keys x 64 dims (rows beyond T are zero)
    for (int u = tid; u < AKC * 8; u += 256) {
      const int r = u >> 3, cc = (u & 7) * 8;
      const int key = ch * AKC + r;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (key < Tn) v = *(const uint4*)(kg + (size_t)key * ld + cc);
      *(uint4*)(Ks + r * AKS + cc) = v;
    }
    __syncthreads();
#pragma unroll
    for (int t = 0; t < MAXT; t++) {
      if ((t >> 2) == ch) {
        const bf16_t* kr = Ks + ((t & 3) * 16 + c) * AKS + 8 * g;
        const bf16x8_t k0 = *(const bf16x8_t*)kr;
        const bf16x8_t k1 = *(const bf16x8_t*)(kr + 32);
        S[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qop[0], S[t], 0, 0, 0);
        S[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qop[1], S[t], 0, 0, 0);
      }
    }
  }

  // ---- softmax with the exact row maximum (lane's query = q0 + c)
  float mx = -INFINITY;
#pragma unroll
  for (int t = 0; t < MAXT; t++) {
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int key = t * 16 + 4 * g + j;
      float v = -INFINITY;
        if (t < nkt && key < Tn) v = fmaf(S[t][j], sc2, lnS[key]);
      S[t][j] = v;
      mx = fmaxf(mx, v);
    }
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
  float ls = 0.f;
#pragma unroll
  for (int t = 0; t < MAXT; t++)
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const float e = (t < nkt) ? __builtin_amdgcn_exp2f(S[t][j] - mx) : 0.f;
      S[t][j] = e;
      ls += e;
    }
  ls += __shfl_xor(ls, 16, 64);
  ls += __shfl_xor(ls, 32, 64);
  const float rl = 1.0f / ls;

  if (a.cls_scores && q0 == 0 && c == 0) {
    float* cs = a.cls_scores + ((size_t)i * a.H + h) * a.tmax;
#pragma unroll
    for (int t = 0; t < MAXT; t++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const int key = t * 16 + 4 * g + j;
        if (t < nkt && key < Tn) cs[key] = S[t][j] * rl;
      }
  }

  // ---- phase 2: O = round(E) V over key-tile pairs
  f32x4_t O[4];
#pragma unroll
  for (int n = 0; n < 4; n++) O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  const bf16_t* vg = qkv + (size_t)base * ld + 2 * d + h * 64;
  for (int ch = 0; ch < nch; ch++) {
    __syncthreads();
    // stage V^T for 64 keys: Vt[dim][key]; keys beyond T are zero
    for (int u = tid; u < AKC * 8; u += 256) {
      const int r = u >> 3, cc = (u & 7) * 8;
      const int key = ch * AKC + r;
      uint4 v = make_uint4(0, 0, 0, 0);
      if (key < Tn) v = *(const uint4*)(vg + (size_t)key * ld + cc);
      const bf16_t* e = (const bf16_t*)&v;
#pragma unroll
      for (int q = 0; q < 8; q++) Vt[(cc + q) * AVS + r] = e[q];
    }
    __syncthreads();
#pragma unroll
    for (int p = 0; p < (MAXT + 1) / 2; p++) {
      if ((p >> 1) == ch) {
        const int t0 = 2 * p, t1 = 2 * p + 1;
        bf16x8_t pa;
#pragma unroll
        for (int j = 0; j < 4; j++) {
          pa[j] = (__bf16)0.f;
          pa[4 + j] = (__bf16)0.f;
        }
        {
          union { bf16_t u[8]; bf16x8_t v; } cv;
#pragma unroll
          for (int j = 0; j < 4; j++) {
            cv.u[j] = f32_to_bf16(t0 < MAXT ? S[t0 < MAXT ? t0 : 0][j] : 0.f);
            cv.u[4 + j] = f32_to_bf16(t1 < MAXT ? S[t1 < MAXT ? t1 : 0][j] : 0.f);
          }
          pa = cv.v;
        }
        const int kl = (p & 1) * 32 + 4 * g;  // key offset inside the chunk
#pragma unroll
        for (int n = 0; n < 4; n++) {
          const bf16_t* vr = Vt + (n * 16 + c) * AVS + kl;
          union { uint2 u[2]; bf16x8_t v; } vb;
          vb.u[0] = *(const uint2*)vr;
          vb.u[1] = *(const uint2*)(vr + 16);
          O[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa, vb.v, O[n], 0, 0, 0);
        }
      }
    }
  }

  // ---- normalise and store: lane holds O[q0 + 4g + j][16n + c]
  bf16_t* out = (bf16_t*)a.out;
#pragma unroll
  for (int j = 0; j < 4; j++) {
    const int q = q0 + 4 * g + j;
    const float l = __shfl(rl, 4 * g + j, 64);
    if (q < Tn) {
#pragma unroll
      for (int n = 0; n < 4; n++)
        out[(size_t)(base + q) * d + h * 64 + n * 16 + c] = f32_to_bf16(O[n][j] * l);
    }
  }
}

// Resident variant for T <= 16 * MAXT <= 256 keys: one workgroup per (live
// sample, head) stages K (padded rows) and V^T ([dim][key], built with an
// 8x8 register transpose and 16-byte LDS stores) once; then each wave walks
// the query tiles qt = wave, wave + 4, ... with no further barrier.  Per
// query tile the arithmetic is the chunked kernel's: transposed scores with
// the exact row maximum, then round(E) V with the key permutation.
constexpr int RKS = 64 + 8;  // K row stride (bf16)

template <int MAXT>
__global__ __launch_bounds__(256) void attention_mfma_res(AttnArgs a) {
  constexpr int TP = MAXT * 16;      // padded keys
  constexpr int TPE = ((MAXT + 1) / 2) * 32;  // keys covered by tile pairs
  constexpr int VTS = TPE + 8;       // V^T row stride (bf16)
  const int i = blockIdx.x, h = blockIdx.y;
  if (i >= a.cnt->nlive) return;
  const int base = a.cu[i], Tn = a.cu[i + 1] - base;
  if (Tn > a.T_ub || Tn > TP) return;  // the host bound is exact
  if (h == 0 && threadIdx.x == 0 && a.token_counts)
    a.token_counts[a.live[i] * a.L + a.b0] = Tn;
  const int d = a.d, ld = 3 * d;
  const float sc2 = a.scale * kLog2e;
  const bf16_t* qkv = (const bf16_t*)a.qkv;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[TP * RKS];
  __shared__ __attribute__((aligned(16))) bf16_t Vt[64 * VTS];
  __shared__ float lnS[TP];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c = lane & 15;
  const int nkt = (Tn + 15) >> 4;

  // ---- staging: every global load (K rows, V rows, token sizes) is issued
  // before the first LDS write, so the workgroup waits for one memory
  // latency instead of one per loop trip
  static_assert(MAXT <= 16, "one V block and one size per thread");
  constexpr int KU = (TP * 8 + 255) / 256;  // 16-byte K pieces per thread
  const bf16_t* kg = qkv + (size_t)base * ld + d + h * 64;
  const bf16_t* vg = qkv + (size_t)base * ld + 2 * d + h * 64;
  const int nkt2 = (nkt + 1) & ~1;
  uint4 kin[KU];
#pragma unroll
  for (int w = 0; w < KU; w++) {
    const int u = tid + w * 256;
    const int r = u >> 3, cc = (u & 7) * 8;
    kin[w] = make_uint4(0, 0, 0, 0);
    if (u < nkt * 16 * 8 && r < Tn) kin[w] = *(const uint4*)(kg + (size_t)r * ld + cc);
  }
  // V^T: thread = 8 keys x 8 dims block, transposed in registers; staged up
  // to an even number of key tiles (zeros past T), so the last tile pair of
  // P V never reads outside the staged keys
  const int kb = tid >> 3, db = (tid & 7) * 8;   // keys 8kb.., dims db..
  const bool vth = tid < nkt2 * 2 * 8;
  uint32_t in[8][4];
#pragma unroll
  for (int r = 0; r < 8; r++) {
    uint4 v = make_uint4(0, 0, 0, 0);
    if (vth && kb * 8 + r < Tn) v = *(const uint4*)(vg + (size_t)(kb * 8 + r) * ld + db);
    in[r][0] = v.x; in[r][1] = v.y; in[r][2] = v.z; in[r][3] = v.w;
  }
  const bool sth = tid < nkt * 16;
  const float sz = (sth && tid < Tn && a.prop_attn) ? a.size[base + tid] : 1.f;
#pragma unroll
  for (int w = 0; w < KU; w++) {
    const int u = tid + w * 256;
    if (u < nkt * 16 * 8) *(uint4*)(Ks + (u >> 3) * RKS + (u & 7) * 8) = kin[w];
  }
  if (vth) {
#pragma unroll
    for (int j = 0; j < 8; j++) {
      uint32_t w[4];
#pragma unroll
      for (int q = 0; q < 4; q++) {
        const uint32_t lo = (in[2 * q][j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
        const uint32_t hi = (in[2 * q + 1][j >> 1] >> (16 * (j & 1))) & 0xFFFFu;
        w[q] = lo | (hi << 16);
      }
      *(uint4*)(Vt + (db + j) * VTS + kb * 8) = make_uint4(w[0], w[1], w[2], w[3]);
    }
  }
  if (sth) lnS[tid] = (tid < Tn && a.prop_attn) ? logf(sz) * kLog2e : 0.f;
  __syncthreads();

  bf16_t* out = (bf16_t*)a.out;
  // Q^T operand of the wave's first query tile; the next tile's is fetched
  // while the current one is processed
  uint4 qnext[2];
  auto load_q = [&](int qt, uint4* dstq) {
    const int q = qt * 16 + c;
    const bf16_t* qr = qkv + (size_t)(base + q) * ld + h * 64;
#pragma unroll
    for (int hf = 0; hf < 2; hf++)
      dstq[hf] = (q < Tn) ? *(const uint4*)(qr + hf * 32 + 8 * g) : make_uint4(0, 0, 0, 0);
  };
  load_q(wave, qnext);
  for (int qt = wave; qt < nkt; qt += 4) {
    const int q0 = qt * 16;
    bf16x8_t qop[2];
    qop[0] = *(bf16x8_t*)&qnext[0];
    qop[1] = *(bf16x8_t*)&qnext[1];
    if (qt + 4 < nkt) load_q(qt + 4, qnext);
    f32x4_t S[MAXT];
#pragma unroll
    for (int t = 0; t < MAXT; t++) {
      S[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
      if (t < nkt) {
        const bf16_t* kr = Ks + (t * 16 + c) * RKS + 8 * g;
        const bf16x8_t k0 = *(const bf16x8_t*)kr;
        const bf16x8_t k1 = *(const bf16x8_t*)(kr + 32);
        S[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qop[0], S[t], 0, 0, 0);
        S[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qop[1], S[t], 0, 0, 0);
      }
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < MAXT; t++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const int key = t * 16 + 4 * g + j;
        float v = -INFINITY;
        if (t < nkt && key < Tn) v = fmaf(S[t][j], sc2, lnS[key]);
        S[t][j] = v;
        mx = fmaxf(mx, v);
      }
    mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    float ls = 0.f;
#pragma unroll
    for (int t = 0; t < MAXT; t++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const float e = (t < nkt) ? __builtin_amdgcn_exp2f(S[t][j] - mx) : 0.f;
        S[t][j] = e;
        ls += e;
      }
    ls += __shfl_xor(ls, 16, 64);
    ls += __shfl_xor(ls, 32, 64);
    const float rl = 1.0f / ls;
    if (a.cls_scores && q0 == 0 && c == 0) {
      float* cs = a.cls_scores + ((size_t)i * a.H + h) * a.tmax;
#pragma unroll
      for (int t = 0; t < MAXT; t++)
#pragma unroll
        for (int j = 0; j < 4; j++) {
          const int key = t * 16 + 4 * g + j;
          if (t < nkt && key < Tn) cs[key] = S[t][j] * rl;
        }
    }
    f32x4_t O[4];
#pragma unroll
    for (int n = 0; n < 4; n++) O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int p = 0; p < (MAXT + 1) / 2; p++) {
      const int t0 = 2 * p, t1 = 2 * p + 1;
      if (t0 < nkt) {
        union { bf16_t u[8]; bf16x8_t v; } cv;
#pragma unroll
        for (int j = 0; j < 4; j++) {
          cv.u[j] = f32_to_bf16(S[t0][j]);
          cv.u[4 + j] = (t1 < MAXT) ? f32_to_bf16(S[t1 < MAXT ? t1 : 0][j]) : (bf16_t)0;
        }
        const int kl = 32 * p + 4 * g;
#pragma unroll
        for (int n = 0; n < 4; n++) {
          const bf16_t* vr = Vt + (n * 16 + c) * VTS + kl;
          union { uint2 u[2]; bf16x8_t v; } vb;
          vb.u[0] = *(const uint2*)vr;
          vb.u[1] = *(const uint2*)(vr + 16);
          O[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cv.v, vb.v, O[n], 0, 0, 0);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int q = q0 + 4 * g + j;
      const float l = __shfl(rl, 4 * g + j, 64);
      if (q < Tn) {
#pragma unroll
        for (int n = 0; n < 4; n++)
          out[(size_t)(base + q) * d + h * 64 + n * 16 + c] = f32_to_bf16(O[n][j] * l);
      }
    }
  }
}

template <typename T>
hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.nlive_ub <= 0) return hipSuccess;
  if (sizeof(T) == 2 && a.dh == 64) {
    if (a.T_ub <= 16 * 13) {
      attention_mfma_res<13><<<dim3(a.nlive_ub, a.H), 256, 0, s>>>(a);
      return hipGetLastError();
    }
    if (a.T_ub <= 16 * 16) {
      attention_mfma_res<16><<<dim3(a.nlive_ub, a.H), 256, 0, s>>>(a);
      return hipGetLastError();
    }
    dim3 grid(a.nlive_ub, a.H, (a.T_ub + 63) / 64);
    if (a.T_ub <= 16 * 40)
      attention_mfma<40><<<grid, 256, 0, s>>>(a);
    else
      return hipErrorInvalidValue;
    return hipGetLastError();
  }
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
