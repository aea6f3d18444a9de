// Multi-head self-attention over ragged samples (Eq. 2), with proportional
// attention (scores += ln of the key token's size) and, on prune blocks, the
// per-head CLS attention row that scores tokens for pruning.
//
// Softmax uses the exact row maximum: the full score row of a query is held
// (LDS or registers) before exponentiation, or, in the chunked MFMA kernel
// for long samples, found by a first pass over the keys whose scores the
// second pass recomputes bit for bit.  E = exp(S - max), l = sum E in
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
// any length up to 16 * MAXT keys fits: one pass over the chunks for the
// row maximum, a second for E, l and O.  For O = P V the lane's own
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
constexpr int AVS = AKC + 4;       // V^T chunk row stride (bf16): an odd multiple of 8 bytes

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

  // Two passes over the key chunks, each holding one chunk's scores in
  // registers (a whole score row would take 160 VGPRs at 640 keys and leave
  // one wave per SIMD): the first finds the exact row maximum, the second
  // recomputes the same scores (same MFMA operands and order, so the same
  // bits), exponentiates them and accumulates l and round(E) V chunk by
  // chunk in the key order of a single pass.
  const bf16_t* kg = qkv + (size_t)base * ld + d + h * 64;
  const bf16_t* vg = qkv + (size_t)base * ld + 2 * d + h * 64;
  // stage 64 keys x 64 dims of K, and optionally V^T ([dim][key]); rows
  // beyond T are zero.  The global loads of a chunk (load) are issued one
  // chunk ahead into registers and written to LDS (put) after the barrier
  // that ends the previous chunk's reads.
  constexpr int SW = AKC * 8 / 256;  // 16-byte pieces per thread and chunk
  auto load = [&](int ch, bool with_v, uint4* kv, uint4* vv) {
#pragma unroll
    for (int w = 0; w < SW; w++) {
      const int u = tid + w * 256;
      const int key = ch * AKC + (u >> 3), cc = (u & 7) * 8;
      kv[w] = make_uint4(0, 0, 0, 0);
      vv[w] = make_uint4(0, 0, 0, 0);
      if (key < Tn) {
        kv[w] = *(const uint4*)(kg + (size_t)key * ld + cc);
        if (with_v) vv[w] = *(const uint4*)(vg + (size_t)key * ld + cc);
      }
    }
  };
  auto put = [&](bool with_v, const uint4* kv, const uint4* vv) {
#pragma unroll
    for (int w = 0; w < SW; w++) {
      const int u = tid + w * 256;
      const int r = u >> 3, cc = (u & 7) * 8;
      *(uint4*)(Ks + r * AKS + cc) = kv[w];
      if (with_v) {
        const bf16_t* e = (const bf16_t*)&vv[w];
#pragma unroll
        for (int q = 0; q < 8; q++) Vt[(cc + q) * AVS + r] = e[q];
      }
    }
  };
  // base-2 scores of the chunk's four key tiles: lane (g, c) holds keys
  // 16t + 4g + j of query q0 + c, with the key term; -inf past the keys
  auto scores = [&](int ch, f32x4_t* s4) {
#pragma unroll
    for (int tt = 0; tt < 4; tt++) {
      const int t = 4 * ch + tt;
      f32x4_t sv = f32x4_t{0.f, 0.f, 0.f, 0.f};
      if (t < MAXT) {
        const bf16_t* kr = Ks + (tt * 16 + c) * AKS + 8 * g;
        const bf16x8_t k0 = *(const bf16x8_t*)kr;
        const bf16x8_t k1 = *(const bf16x8_t*)(kr + 32);
        sv = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k0, qop[0], sv, 0, 0, 0);
        sv = __builtin_amdgcn_mfma_f32_16x16x32_bf16(k1, qop[1], sv, 0, 0, 0);
      }
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const int key = t * 16 + 4 * g + j;
        float v = -INFINITY;
        if (t < nkt && key < Tn) v = fmaf(sv[j], sc2, lnS[key]);
        s4[tt][j] = v;
      }
    }
  };

  // ---- pass 1: the exact row maximum
  float mx = -INFINITY;
  uint4 kv[SW], vv[SW];
  load(0, false, kv, vv);
  for (int ch = 0; ch < nch; ch++) {
    __syncthreads();
    put(false, kv, vv);
    __syncthreads();
    if (ch + 1 < nch) load(ch + 1, false, kv, vv);
    f32x4_t s4[4];
    scores(ch, s4);
#pragma unroll
    for (int tt = 0; tt < 4; tt++)
#pragma unroll
      for (int j = 0; j < 4; j++) mx = fmaxf(mx, s4[tt][j]);
  }
  mx = fmaxf(mx, __shfl_xor(mx, 16, 64));
  mx = fmaxf(mx, __shfl_xor(mx, 32, 64));

  // ---- pass 2: E = exp2(s - max), l = sum E, O = round(E) V over key-tile
  // pairs; the CLS query's E go out unnormalised and are scaled by 1 / l
  // once l is known
  const bool cls_lane = a.cls_scores && q0 == 0 && c == 0;
  float* cs = a.cls_scores ? a.cls_scores + ((size_t)i * a.H + h) * a.tmax : nullptr;
  float ls = 0.f;
  f32x4_t O[4];
#pragma unroll
  for (int n = 0; n < 4; n++) O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  load(0, true, kv, vv);
  for (int ch = 0; ch < nch; ch++) {
    __syncthreads();
    put(true, kv, vv);
    __syncthreads();
    if (ch + 1 < nch) load(ch + 1, true, kv, vv);
    f32x4_t s4[4];
    scores(ch, s4);
#pragma unroll
    for (int tt = 0; tt < 4; tt++) {
      const int t = 4 * ch + tt;
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const float e = (t < nkt) ? __builtin_amdgcn_exp2f(s4[tt][j] - mx) : 0.f;
        s4[tt][j] = e;
        ls += e;
        const int key = t * 16 + 4 * g + j;
        if (cls_lane && t < nkt && key < Tn) cs[key] = e;
      }
    }
#pragma unroll
    for (int pp = 0; pp < 2; pp++) {
      const int p = 2 * ch + pp, t1 = 2 * p + 1;
      if (p < (MAXT + 1) / 2) {
        union { bf16_t u[8]; bf16x8_t v; } cv;
#pragma unroll
        for (int j = 0; j < 4; j++) {
          cv.u[j] = f32_to_bf16(s4[2 * pp][j]);
          cv.u[4 + j] = f32_to_bf16(t1 < MAXT ? s4[2 * pp + 1][j] : 0.f);
        }
        const int kl = pp * 32 + 4 * g;  // key offset inside the chunk
#pragma unroll
        for (int n = 0; n < 4; n++) {
          const bf16_t* vr = Vt + (n * 16 + c) * AVS + kl;
          union { uint2 u[2]; bf16x8_t v; } vb;
          vb.u[0] = *(const uint2*)vr;
          vb.u[1] = *(const uint2*)(vr + 16);
          O[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cv.v, vb.v, O[n], 0, 0, 0);
        }
      }
    }
  }
  ls += __shfl_xor(ls, 16, 64);
  ls += __shfl_xor(ls, 32, 64);
  const float rl = 1.0f / ls;
  if (cls_lane) {
    for (int t = 0; t < nkt; t++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const int key = t * 16 + 4 * g + j;
        if (key < Tn) cs[key] = cs[key] * rl;
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
// sample, head) stages K and V (both row-major, [key][dim], with 16-byte
// LDS stores) once; then each of its 8 waves walks the query tiles qt =
// wave, wave + 8, ... with no further barrier.  Per query tile the
// arithmetic is the chunked kernel's: transposed scores with the exact row
// maximum, then round(E) V with the key permutation.
//
// K rows are stored unpadded (128 bytes) with their eight 16-byte chunks
// XOR-permuted by row % 8, so the per-lane 16-byte reads of 16 rows are
// free of bank conflicts.  V rows are unpadded with their four 32-byte
// segments XOR-permuted by (row / 2) % 2, and the V^T operand of the output
// product is read from them with gfx950's transposing LDS read
// (ds_read_b64_tr_b16: within each group of 16 lanes, lane i reads 4
// consecutive 16-bit values, and lane o receives value o % 4 of lanes o / 4,
// o / 4 + 4, o / 4 + 8 and o / 4 + 12), so no register transpose is needed.
//
// The key loops run over all MAXT tiles with no per-tile condition: past
// the sample's T keys, K and V hold finite copies of its last row and the
// additive key term is -inf (so those probabilities are exactly 0 and the
// copies add exact zeros).  The host picks MAXT =
// ceil(T_ub / 16), so at most the tiles between T and the bound are idle.
// The output product is taken transposed (V^T . E^T), so a lane holds four
// consecutive head dimensions of one query and stores them as 8 bytes.
constexpr int RES_NT = 512;  // 8 waves share the staged K and V
// 16-byte staging piece (a vector value, so the staging arrays stay in registers)
typedef unsigned u32x4v __attribute__((ext_vector_type(4)));

// Long samples (17 .. 37 key tiles, T <= 592: the 384 x 384 workload) use
// the same kernel with one workgroup per CU: K (74 KB) and V (76 KB) of the
// (sample, head) fill the LDS, each wave holds a whole score row of its query
// tile in registers (2 waves per SIMD, up to 256 VGPRs), and the staging
// loops cover more keys than threads.
constexpr int RES_LONG_MAXT = 37;

template <int MAXT>
__global__ __launch_bounds__(RES_NT, MAXT <= 16 ? 4 : 1) void attention_mfma_res(AttnArgs a) {
  static_assert(MAXT >= 1 && MAXT <= RES_LONG_MAXT, "resident key range");
  constexpr bool LONG = MAXT > 16;
  constexpr int TP = MAXT * 16;               // padded keys
  constexpr int NP = (MAXT + 1) / 2;          // key tile pairs
  constexpr int TPE = NP * 32;                // keys covered by tile pairs (V rows)
  const int i = blockIdx.x, h = blockIdx.y;
  if (i >= a.cnt->nlive) return;
  const int base = a.cu[i], Tn = a.cu[i + 1] - base;
  if (Tn > a.T_ub || Tn > TP) return;  // the host bound is exact
  if (h == 0 && threadIdx.x == 0 && a.token_counts)
    a.token_counts[a.live[i] * a.L + a.b0] = Tn;
  const int d = a.d, ld = 3 * d;
  const float sc2 = a.scale * kLog2e;
  const bf16_t* qkv = (const bf16_t*)a.qkv;
  __shared__ __attribute__((aligned(16))) bf16_t Ks[TP * 64];
  __shared__ __attribute__((aligned(16))) bf16_t Vs[TPE * 64];
  __shared__ __attribute__((aligned(16))) float lnS[TP];
  __shared__ __attribute__((aligned(16))) float clsP[TP];
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c = lane & 15;
  const int nkt = (Tn + 15) >> 4;

  // ---- staging: every global load (K rows, V rows, token sizes) is issued
  // before the first LDS write, so the workgroup waits for one memory
  // latency instead of one per loop trip
  constexpr int KU = (TP * 8 + RES_NT - 1) / RES_NT;  // 16-byte K pieces per thread
  const bf16_t* kg = qkv + (size_t)base * ld + d + h * 64;
  const bf16_t* vg = qkv + (size_t)base * ld + 2 * d + h * 64;
  // (rows past the sample read its last row, so no load sits behind a
  // branch and they issue together; those keys keep these finite copies,
  // whose probabilities are exactly 0 since their key term is -inf)
  u32x4v kin[KU];
#pragma unroll
  for (int w = 0; w < KU; w++) {
    const int u = tid + w * RES_NT;
    const int r = u >> 3, cc = (u & 7) * 8;
    kin[w] = *(const u32x4v*)(kg + (size_t)min(r, Tn - 1) * ld + cc);
  }
  constexpr int VU = (TPE * 8 + RES_NT - 1) / RES_NT;  // 16-byte V pieces per thread
  u32x4v vin[VU];
#pragma unroll
  for (int w = 0; w < VU; w++) {
    const int u = tid + w * RES_NT;
    const int r = u >> 3, cc = (u & 7) * 8;
    vin[w] = *(const u32x4v*)(vg + (size_t)min(r, Tn - 1) * ld + cc);
  }
  constexpr int SR = LONG ? (TP + RES_NT - 1) / RES_NT : 1;  // sizes per thread
  float szr[SR];
#pragma unroll
  for (int v = 0; v < SR; v++) szr[v] = a.size[base + min(tid + v * RES_NT, Tn - 1)];
  __builtin_amdgcn_sched_barrier(0);  // every load above is in flight before any use
#pragma unroll
  for (int w = 0; w < KU; w++) {
    const int u = tid + w * RES_NT;
    if (u < TP * 8)
      *(u32x4v*)(Ks + (u >> 3) * 64 + (((u & 7) ^ ((u >> 3) & 7)) << 3)) = kin[w];
  }
#pragma unroll
  for (int w = 0; w < VU; w++) {
    const int u = tid + w * RES_NT;
    const int r = u >> 3;
    if (u < TPE * 8)
      *(u32x4v*)(Vs + r * 64 + (((u & 7) ^ (((r >> 1) & 1) << 1)) << 3)) = vin[w];
  }
  // key term of the base-2 scores: log2(size) (0 without proportional
  // attention), -inf past the sample's keys
#pragma unroll
  for (int v = 0; v < SR; v++) {
    const int t = tid + v * RES_NT;
    const float sz = (t < Tn && a.prop_attn) ? szr[v] : 1.f;
    if (t < TP) lnS[t] = t < Tn ? logf(sz) * kLog2e : -INFINITY;
  }
  __syncthreads();

  bf16_t* out = (bf16_t*)a.out;
  const bool want_cls = a.cls_scores != nullptr;
  // Q^T operand of the wave's first query tile; the next tile's is fetched
  // while the current one is processed (queries past the sample read its
  // last row: their rows are computed and never stored)
  uint4 qnext[2];
  auto load_q = [&](int qt, uint4* dstq) {
    const int q = min(qt * 16 + c, Tn - 1);
    const bf16_t* qr = qkv + (size_t)(base + q) * ld + h * 64;
#pragma unroll
    for (int hf = 0; hf < 2; hf++) dstq[hf] = *(const uint4*)(qr + hf * 32 + 8 * g);
  };
  load_q(wave, qnext);
  for (int qt = wave; qt < nkt; qt += RES_NT / 64) {
    const int q0 = qt * 16;
    bf16x8_t qop[2];
    qop[0] = *(bf16x8_t*)&qnext[0];
    qop[1] = *(bf16x8_t*)&qnext[1];
    if (qt + RES_NT / 64 < nkt) load_q(qt + RES_NT / 64, qnext);
    // S^T tiles: lane (g, c) holds keys 16t + 4g + j of query q0 + c.  The
    // K operands are read two tiles ahead; the scheduling barriers keep the
    // compiler from hoisting every read (which would exhaust the registers).
    f32x4_t S[MAXT];
    bf16x8_t kf[3][2];
    auto load_k = [&](int t, bf16x8_t* dstk) {
      const int r = t * 16 + c;
      const bf16_t* kr = Ks + r * 64;
      dstk[0] = *(const bf16x8_t*)(kr + ((g ^ (r & 7)) << 3));
      dstk[1] = *(const bf16x8_t*)(kr + (((4 + g) ^ (r & 7)) << 3));
    };
    load_k(0, kf[0]);
    if (MAXT > 1) load_k(1, kf[1]);
#pragma unroll
    for (int t = 0; t < MAXT; t++) {
      if (t + 2 < MAXT) load_k(t + 2, kf[(t + 2) % 3]);
      S[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[t % 3][0], qop[0],
                                                      f32x4_t{0.f, 0.f, 0.f, 0.f}, 0, 0, 0);
      S[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[t % 3][1], qop[1], S[t], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    float mx = -INFINITY;
#pragma unroll
    for (int t = 0; t < MAXT; t++) {
      const float4 ks = *(const float4*)(lnS + t * 16 + 4 * g);
      S[t][0] = fmaf(S[t][0], sc2, ks.x);
      S[t][1] = fmaf(S[t][1], sc2, ks.y);
      S[t][2] = fmaf(S[t][2], sc2, ks.z);
      S[t][3] = fmaf(S[t][3], sc2, ks.w);
      mx = fmaxf(mx, fmaxf(fmaxf(S[t][0], S[t][1]), fmaxf(S[t][2], S[t][3])));
    }
    mx = max_xor32(max_xor16(mx));
    float ls = 0.f;
#pragma unroll
    for (int t = 0; t < MAXT; t++)
#pragma unroll
      for (int j = 0; j < 4; j++) {
        const float e = __builtin_amdgcn_exp2f(S[t][j] - mx);
        S[t][j] = e;
        ls += e;
      }
    ls = sum_xor32(sum_xor16(ls));
    const float rl = 1.0f / ls;
    if (want_cls && q0 == 0 && c == 0) {
#pragma unroll
      for (int t = 0; t < MAXT; t++)
        *(float4*)(clsP + t * 16 + 4 * g) =
            make_float4(S[t][0] * rl, S[t][1] * rl, S[t][2] * rl, S[t][3] * rl);
    }
    // O^T = V^T . E^T: lane (g, c) accumulates dims 16n + 4g + j of query q0 + c
    f32x4_t O[4];
#pragma unroll
    for (int n = 0; n < 4; n++) O[n] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // V^T operand of key pair p, dims 16n ..: lane (g, c) needs keys
    // 32p + 4g + 0..3 and 32p + 16 + 4g + 0..3 of dim 16n + c; with the
    // transposing read, lane c of the group reads dims 16n + 4(c % 4) .. + 3
    // of key Kb + c / 4 (Kb = 32p + 4g, then Kb + 16).  (Kb / 2 is even, so
    // the key's segment permutation bit is (c / 8) % 2.)
    union VB { uint2 u[2]; bf16x8_t v; };
    VB vb[2][4];
    const int vsb = (c >> 3) & 1;
    const char* vlane = (const char*)Vs + (4 * g + (c >> 2)) * 128 + 8 * (c & 3);
    auto load_v = [&](int p, VB* dstv) {
#pragma unroll
      for (int n = 0; n < 4; n++)
#pragma unroll
        for (int hh = 0; hh < 2; hh++) {
          typedef short v4s __attribute__((ext_vector_type(4)));
          const char* pa = vlane + (32 * p + 16 * hh) * 128 + ((n ^ vsb) << 5);
          const v4s r = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
              (__attribute__((address_space(3))) v4s*)pa);
          dstv[n].u[hh] = __builtin_bit_cast(uint2, r);
        }
    };
    load_v(0, vb[0]);
#pragma unroll
    for (int p = 0; p < NP; p++) {
      const int t0 = 2 * p, t1 = 2 * p + 1;
      if (p + 1 < NP) load_v(p + 1, vb[(p + 1) & 1]);
      union { uint32_t u[4]; bf16x8_t v; } cv;
      cv.u[0] = pack_bf16x2(S[t0][0], S[t0][1]);
      cv.u[1] = pack_bf16x2(S[t0][2], S[t0][3]);
      if (t1 < MAXT) {
        cv.u[2] = pack_bf16x2(S[t1 < MAXT ? t1 : 0][0], S[t1 < MAXT ? t1 : 0][1]);
        cv.u[3] = pack_bf16x2(S[t1 < MAXT ? t1 : 0][2], S[t1 < MAXT ? t1 : 0][3]);
      } else {
        cv.u[2] = 0u;
        cv.u[3] = 0u;
      }
#pragma unroll
      for (int n = 0; n < 4; n++)
        O[n] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vb[p & 1][n].v, cv.v, O[n], 0, 0, 0);
      __builtin_amdgcn_sched_barrier(0);
    }
    const int q = q0 + c;
    if (q < Tn) {
      bf16_t* orow = out + (size_t)(base + q) * d + h * 64 + 4 * g;
#pragma unroll
      for (int n = 0; n < 4; n++) {
        *(uint2*)(orow + n * 16) = make_uint2(pack_bf16x2(O[n][0] * rl, O[n][1] * rl),
                                              pack_bf16x2(O[n][2] * rl, O[n][3] * rl));
      }
    }
  }
  // CLS-query probabilities of this head (prune blocks), copied out by the
  // whole workgroup once wave 0 has written them
  if (want_cls) {
    __syncthreads();
    float* cs = a.cls_scores + ((size_t)i * a.H + h) * a.tmax;
    for (int k = tid; k < Tn; k += RES_NT) cs[k] = clsP[k];
  }
}

template <typename T>
hipError_t launch_attention(const AttnArgs& a, hipStream_t s) {
  if (a.nlive_ub <= 0) return hipSuccess;
  if (sizeof(T) == 2 && a.dh == 64) {
    if (a.T_ub <= 16 * 16) {
      const dim3 grid(a.nlive_ub, a.H);
      switch ((a.T_ub + 15) / 16) {
#define FUSION_ATTN_RES(n) \
  case n: attention_mfma_res<n><<<grid, RES_NT, 0, s>>>(a); break;
        FUSION_ATTN_RES(1) FUSION_ATTN_RES(2) FUSION_ATTN_RES(3) FUSION_ATTN_RES(4)
        FUSION_ATTN_RES(5) FUSION_ATTN_RES(6) FUSION_ATTN_RES(7) FUSION_ATTN_RES(8)
        FUSION_ATTN_RES(9) FUSION_ATTN_RES(10) FUSION_ATTN_RES(11) FUSION_ATTN_RES(12)
        FUSION_ATTN_RES(13) FUSION_ATTN_RES(14) FUSION_ATTN_RES(15) FUSION_ATTN_RES(16)
        default: return hipErrorInvalidValue;
      }
      return hipGetLastError();
    }
    if (a.T_ub <= 16 * RES_LONG_MAXT) {
      const dim3 grid(a.nlive_ub, a.H);
      switch ((a.T_ub + 15) / 16) {
        FUSION_ATTN_RES(17) FUSION_ATTN_RES(18) FUSION_ATTN_RES(19) FUSION_ATTN_RES(20)
        FUSION_ATTN_RES(21) FUSION_ATTN_RES(22) FUSION_ATTN_RES(23) FUSION_ATTN_RES(24)
        FUSION_ATTN_RES(25) FUSION_ATTN_RES(26) FUSION_ATTN_RES(27) FUSION_ATTN_RES(28)
        FUSION_ATTN_RES(29) FUSION_ATTN_RES(30) FUSION_ATTN_RES(31) FUSION_ATTN_RES(32)
        FUSION_ATTN_RES(33) FUSION_ATTN_RES(34) FUSION_ATTN_RES(35) FUSION_ATTN_RES(36)
        FUSION_ATTN_RES(37)
        default: return hipErrorInvalidValue;
      }
      return hipGetLastError();
    }
#undef FUSION_ATTN_RES
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
