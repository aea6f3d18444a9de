// Per-sample adaptive steps after a block (Algorithm 1, Sec. III-B..E):
//   merge router and count (Eq. 4-5), bipartite soft matching with
//   size-weighted merging (Sec. III-C), exit check on the CLS head
//   (Eq. 6-7), CLS-attention top-k pruning of continuing samples (Eq. 8),
// followed by a separate compaction kernel that re-packs the surviving
// samples and tokens (exclusive scans over new lengths and keep flags).
//
// One 512-thread workgroup per live sample (the compaction uses 256).  No
// float atomics: every reduction has a fixed order, so results do not depend
// on scheduling or on the rest of the batch.
#include "kernels.h"

namespace fusion {

constexpr int AD_TMAX = 640;  // tokens per sample (CLS included), largest size class
constexpr int AD_NT = 512;    // threads per workgroup (8 waves)
constexpr int SAG = 128;      // A rows per pass: one 16-row MFMA tile per wave

// Size classes of the per-sample kernel: TMAX tokens (CLS included), so
// |A| = ceil(N/2) and |B| = floor(N/2) are at most TMAX/2; the similarity
// features are staged in chunks of SKC (64 for the small class: fewer
// round trips to memory; 32 for the large one, whose B tiles fill the LDS).
template <int TMAX_> struct AdSize {
  static constexpr int TMAX = TMAX_;
  static constexpr int AMAX = TMAX_ / 2;
  static constexpr int BMAX = TMAX_ / 2;
  static constexpr int SKC = TMAX_ <= 256 ? 64 : 32;
  static constexpr int SKP = SKC + 8;          // padded LDS row (bf16)
  static constexpr int NBT = BMAX / 16;        // B tiles held in registers
  static constexpr int SPT = ((SAG + BMAX) * (SKC / 4) + AD_NT - 1) / AD_NT;  // slots / thread
};

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

__device__ __forceinline__ int merge_count(float m, double rho, int r_b, int N, int rule) {
  // budget:   r = clamp(floor(((2 rho) m) r_b + 1/2), 0, floor(N/2));
  // fraction: r = min(floor(((rho m) N) / 2), floor(N/2)) (Sec. III-C with
  //           the rescaled ratio of Eq. 5);
  // every step an individually rounded IEEE double operation.
  const double t =
      rule == 1 ? __dmul_rn(__dmul_rn(__dmul_rn(rho, (double)m), (double)N), 0.5)
                : __dadd_rn(__dmul_rn(__dmul_rn(__dmul_rn(2.0, rho), (double)m), (double)r_b), 0.5);
  int r = (int)floor(t);
  if (r < 0) r = 0;
  if (r > N / 2) r = N / 2;
  return r;
}

// Block-wide reductions for AD_NT threads (8 waves); red >= 8 entries.
__device__ __forceinline__ float bsum(float v, float* red) {
  v = wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < AD_NT / 64; w++) s += red[w];
  return s;
}
__device__ __forceinline__ float bmax(float v, float* red) {
  v = wave_max(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  float s = red[0];
#pragma unroll
  for (int w = 1; w < AD_NT / 64; w++) s = fmaxf(s, red[w]);
  return s;
}
__device__ __forceinline__ int bsum_i(int v, int* red) {
  v = wave_sum_i(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  int s = 0;
#pragma unroll
  for (int w = 0; w < AD_NT / 64; w++) s += red[w];
  return s;
}

// Stream compaction over the workgroup (one candidate per thread): writes
// the indices `v` of the threads with `f` set to out[0 ..) in thread order
// and returns their count.  red >= AD_NT / 64 ints.
__device__ __forceinline__ int block_compact(bool f, int v, int* out, int* red) {
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const unsigned long long msk = __ballot(f);
  __syncthreads();
  if (lane == 0) red[wave] = __popcll(msk);
  __syncthreads();
  int off = 0, tot = 0;
#pragma unroll
  for (int w = 0; w < AD_NT / 64; w++) {
    off += w < wave ? red[w] : 0;
    tot += red[w];
  }
  if (f) out[off + __popcll(msk & ((1ull << lane) - 1ull))] = v;
  __syncthreads();
  return tot;
}

// Split a float into bf16 hi + lo with hi + lo = v to about 2^-17 relative.
__device__ __forceinline__ void split_bf16(float v, bf16_t& hi, bf16_t& lo) {
  hi = f32_to_bf16(v);
  lo = f32_to_bf16(v - bf16_to_f32(hi));
}

// Cosine similarities of the A tokens (even patch slots) with the B tokens
// (odd slots) of one sample, and the best B for every A.
//
// One pass over the features in chunks of SKC: every thread stages a fixed
// set of (row, 4-feature) slots, splits the fp32 values into bf16 hi + lo,
// and accumulates the row's sum of squares on the way; the dot products
// take hi.hi' + hi.lo' + lo.hi' on v_mfma_f32_16x16x32_bf16 with fp32
// accumulation (absolute error of a cosine <= ~1.2e-5, the dropped lo.lo'
// term included).  The loads of chunk k+1 are issued before the MFMAs of
// chunk k.  At the end the dots are divided by the clamped norms
// max(||x||, 1e-12) of both tokens.  Wave w owns A rows ag + 16w .. +15
// against every B tile; lane l of an output tile holds S[a = 4(l/16) + j]
// [b = l%16].
template <class Z>
__device__ void similarity_argmax(const float* __restrict__ x, int base, int d,
                                  int nA, int nB, float* nrm, float* bestsim,
                                  int* best, bf16_t* Ahi, bf16_t* Alo,
                                  bf16_t* Bhi, bf16_t* Blo) {
  constexpr int SKC = Z::SKC, SKP = Z::SKP, SPT = Z::SPT, NBT = Z::NBT;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c = lane & 15;
  const int nbt = (nB + 15) >> 4;
  const int nslot = (SAG + nbt * 16) * (SKC / 4);
  for (int ag = 0; ag < nA; ag += SAG) {
    // this thread's slots: row r = u / (SKC/4) (A rows first, then B rows)
    const float* srow[SPT];
    float ss[SPT];
#pragma unroll
    for (int w = 0; w < SPT; w++) {
      const int u = tid + w * AD_NT;
      const int r = u / (SKC / 4), q = (u % (SKC / 4)) * 4;
      srow[w] = nullptr;
      ss[w] = 0.f;
      if (u < nslot) {
        if (r < SAG) {
          if (ag + r < nA) srow[w] = x + (size_t)(base + 1 + 2 * (ag + r)) * d + q;
        } else if (r - SAG < nB) {
          srow[w] = x + (size_t)(base + 2 + 2 * (r - SAG)) * d + q;
        }
      }
    }
    float4 cur[SPT];
#pragma unroll
    for (int w = 0; w < SPT; w++)
      cur[w] = srow[w] ? *(const float4*)srow[w] : make_float4(0.f, 0.f, 0.f, 0.f);
    f32x4_t acc[NBT];
#pragma unroll
    for (int t = 0; t < NBT; t++) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    for (int k0 = 0; k0 < d; k0 += SKC) {
      __syncthreads();
#pragma unroll
      for (int w = 0; w < SPT; w++) {
        const int u = tid + w * AD_NT;
        if (u >= nslot) continue;
        const int r = u / (SKC / 4), q = (u % (SKC / 4)) * 4;
        bf16_t* H = r < SAG ? Ahi + r * SKP : Bhi + (r - SAG) * SKP;
        bf16_t* Lo = r < SAG ? Alo + r * SKP : Blo + (r - SAG) * SKP;
        const float4 e = cur[w];
        ss[w] = fmaf(e.x, e.x, ss[w]);
        ss[w] = fmaf(e.y, e.y, ss[w]);
        ss[w] = fmaf(e.z, e.z, ss[w]);
        ss[w] = fmaf(e.w, e.w, ss[w]);
        // hi = RNE(v), lo = RNE(v - hi): four values -> two 8-byte stores
        const uint32_t h01 = pack_bf16x2(e.x, e.y), h23 = pack_bf16x2(e.z, e.w);
        const uint32_t l01 = pack_bf16x2(e.x - __uint_as_float(h01 << 16),
                                         e.y - __uint_as_float(h01 & 0xFFFF0000u));
        const uint32_t l23 = pack_bf16x2(e.z - __uint_as_float(h23 << 16),
                                         e.w - __uint_as_float(h23 & 0xFFFF0000u));
        *(uint2*)(H + q) = make_uint2(h01, h23);
        *(uint2*)(Lo + q) = make_uint2(l01, l23);
      }
      // prefetch the next chunk while this one is multiplied
      if (k0 + SKC < d) {
#pragma unroll
        for (int w = 0; w < SPT; w++)
          if (srow[w]) cur[w] = *(const float4*)(srow[w] + k0 + SKC);
      }
      __syncthreads();
      // 32 features per MFMA; per B tile the products accumulate in feature
      // order, hi.hi' then hi.lo' then lo.hi' within each 32
#pragma unroll
      for (int kk = 0; kk < SKC / 32; kk++) {
        const bf16x8_t ah = *(const bf16x8_t*)(Ahi + (wave * 16 + c) * SKP + 32 * kk + 8 * g);
        const bf16x8_t al = *(const bf16x8_t*)(Alo + (wave * 16 + c) * SKP + 32 * kk + 8 * g);
#pragma unroll
        for (int t = 0; t < NBT; t++) {
          if (t < nbt) {
            const bf16x8_t bh = *(const bf16x8_t*)(Bhi + (t * 16 + c) * SKP + 32 * kk + 8 * g);
            const bf16x8_t bl = *(const bf16x8_t*)(Blo + (t * 16 + c) * SKP + 32 * kk + 8 * g);
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bh, acc[t], 0, 0, 0);
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ah, bl, acc[t], 0, 0, 0);
            acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(al, bh, acc[t], 0, 0, 0);
          }
        }
      }
    }
    // row norms: the SKC/4 threads of a row are adjacent lanes
#pragma unroll
    for (int w = 0; w < SPT; w++) {
      float v = ss[w];
#pragma unroll
      for (int o = 1; o < SKC / 4; o <<= 1) v += __shfl_xor(v, o, 64);
      const int u = tid + w * AD_NT;
      const int r = u / (SKC / 4);
      if (srow[w] && (u % (SKC / 4)) == 0) {
        const int slot = r < SAG ? 2 * (ag + r) : 2 * (r - SAG) + 1;  // patch slot
        nrm[slot] = fmaxf(sqrtf(v), 1e-12f);
      }
    }
    __syncthreads();
    // cosine = dot / (n_a n_b); argmax over B, ties to the lowest B index
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int aa = ag + wave * 16 + 4 * g + j;
      const float na = aa < nA ? nrm[2 * aa] : 1.f;
      float bv = -INFINITY;
      int bi = 0x7fffffff;
#pragma unroll
      for (int t = 0; t < NBT; t++) {
        const int bb = t * 16 + c;
        if (t < nbt && bb < nB) {
          const float v = acc[t][j] / (na * nrm[2 * bb + 1]);
          if (v > bv) {
            bv = v;
            bi = bb;
          }
        }
      }
#pragma unroll
      for (int o = 1; o < 16; o <<= 1) {
        const float ov = __shfl_xor(bv, o, 64);
        const int oi = __shfl_xor(bi, o, 64);
        if (ov > bv || (ov == bv && oi < bi)) {
          bv = ov;
          bi = oi;
        }
      }
      if (c == 0 && aa < nA) {
        bestsim[aa] = bv;
        best[aa] = bi < nB ? bi : 0;  // bi >= nB only with non-finite x
      }
    }
    __syncthreads();
  }
}

template <class Z>
__global__ __launch_bounds__(AD_NT) void adapt_kernel(AdaptArgs a) {
  const int i = blockIdx.x;
  if (i >= a.cnt->nlive) return;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int base = a.cu[i], T = a.cu[i + 1] - base, N = T - 1;
  const int orig = a.live[i];
  const int d = a.d;
  const size_t tr_row = (size_t)(a.b - 1) * a.B + orig;

  constexpr int TMAX = Z::TMAX, AMAX = Z::AMAX, BMAX = Z::BMAX, SKP = Z::SKP;
  __shared__ float sc[TMAX];
  __shared__ float szs[TMAX];
  __shared__ int keepf[TMAX];
  __shared__ float nrm[TMAX];
  __shared__ float bestsim[AMAX];
  __shared__ int best[AMAX];
  __shared__ int chosen[AMAX];
  __shared__ int clist[AMAX];
  __shared__ int cdst[AMAX];
  __shared__ int glead[AMAX];
  __shared__ float tmpf[AMAX];
  __shared__ float tmps[AMAX];
  __shared__ __attribute__((aligned(16))) bf16_t Ahi[SAG * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Alo[SAG * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Bhi[BMAX * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Blo[BMAX * SKP];
  __shared__ float red[16];
  __shared__ int ired[16];

  // CLS-attention scores are gathered here and follow the merge; learned
  // scores are computed after the merge from the merged hidden states
  const bool attnP = a.isP && a.prune_rule == 0;
  for (int t = tid; t < T; t += AD_NT) {
    keepf[t] = 1;
    szs[t] = a.size[base + t];
  }
  if (attnP) {
    for (int t = tid; t < T; t += AD_NT) {
      float s = a.cls_scores[((size_t)i * a.H) * a.tmax + t];
      for (int h = 1; h < a.H; h++) s = s + a.cls_scores[((size_t)i * a.H + h) * a.tmax + t];
      sc[t] = s / (float)a.H;
    }
  }
  __syncthreads();

  // ---------------------------------------------------------- merge --
  int r = 0;
  if (a.isM) {
    float z = 0.f;
    for (int k = tid; k < d; k += AD_NT) z = fmaf(a.router_w[k], a.x[(size_t)base * d + k], z);
    z = bsum(z, red) + a.router_b[0];
    const float m = 1.0f / (1.0f + expf(-z));
    r = merge_count(m, a.rho, a.r_b, N, a.merge_rule);
    if (tid == 0) {
      if (a.tr_r) a.tr_r[tr_row] = r;
      if (a.tr_m) a.tr_m[tr_row] = m;
    }
  }
  const int nA = (N + 1) / 2, nB = N / 2;
  if (r > 0) {
    similarity_argmax<Z>(a.x, base, d, nA, nB, nrm, bestsim, best, Ahi, Alo, Bhi, Blo);
    // top-r of A by best similarity, ties to the lower A slot
    for (int aa = tid; aa < nA; aa += AD_NT) {
      const float v = bestsim[aa];
      int rank = 0;
      for (int a2 = 0; a2 < nA; a2++) {
        const float v2 = bestsim[a2];
        rank += (v2 > v) || (v2 == v && a2 < aa);
      }
      chosen[aa] = rank < r;
    }
    __syncthreads();
    // chosen sources in ascending A slot: clist[0 .. r)
    block_compact(tid < nA && chosen[tid], tid, clist, ired);
    // destination of each; a source leads its group when no earlier chosen
    // source has the same destination.  Groups are merged independently,
    // each summing its sources in ascending A slot.
    for (int q = tid; q < r; q += AD_NT) cdst[q] = best[clist[q]];
    __syncthreads();
    bool lead = false;
    if (tid < r) {
      const int bb = cdst[tid];
      lead = true;
      for (int q2 = 0; q2 < tid; q2++) lead = lead && (cdst[q2] != bb);
    }
    const int ng = block_compact(lead, tid, glead, ired);
    // size-weighted merge into each receiving destination (16-byte pieces)
    const int d4 = d / 4;
    float4* x4 = (float4*)a.x;
    for (int idx = tid; idx < ng * d4; idx += AD_NT) {
      const int k = idx / d4, f = idx - k * d4;
      const int q0 = glead[k], bb = cdst[q0];
      const size_t rowb = (size_t)(base + 2 + 2 * bb);
      const float sb = szs[2 + 2 * bb];
      const float4 xb = x4[rowb * d4 + f];
      float4 num = make_float4(sb * xb.x, sb * xb.y, sb * xb.z, sb * xb.w);
      float den = sb;
      for (int q = q0; q < r; q++) {
        if (cdst[q] != bb) continue;
        const int aa = clist[q];
        const float sa = szs[1 + 2 * aa];
        const float4 xa = x4[(size_t)(base + 1 + 2 * aa) * d4 + f];
        num.x = num.x + sa * xa.x;
        num.y = num.y + sa * xa.y;
        num.z = num.z + sa * xa.z;
        num.w = num.w + sa * xa.w;
        den = den + sa;
      }
      x4[rowb * d4 + f] = make_float4(num.x / den, num.y / den, num.z / den, num.w / den);
    }
    for (int k = tid; k < ng; k += AD_NT) {
      const int q0 = glead[k], bb = cdst[q0];
      float den = szs[2 + 2 * bb];
      float s2 = attnP ? sc[2 + 2 * bb] : 0.f;
      for (int q = q0; q < r; q++) {
        if (cdst[q] != bb) continue;
        den = den + szs[1 + 2 * clist[q]];
        if (attnP) s2 = s2 + sc[1 + 2 * clist[q]];
      }
      tmpf[k] = den;
      tmps[k] = s2;
    }
    __syncthreads();
    for (int k = tid; k < ng; k += AD_NT) {
      const int bb = cdst[glead[k]];
      a.size[base + 2 + 2 * bb] = tmpf[k];
      if (attnP) sc[2 + 2 * bb] = tmps[k];
    }
    for (int q = tid; q < r; q += AD_NT) {
      const int aa = clist[q];
      keepf[1 + 2 * aa] = 0;
      if (a.tr_merge)
        a.tr_merge[tr_row * (a.n0 + 1) + a.origin[base + 1 + 2 * aa]] =
            a.origin[base + 2 + 2 * best[aa]];
    }
    __syncthreads();
  }

  // ------------------------------------------------------------ exit --
  bool fire = false;
  if (a.isE) {
    const float* lg = a.head_buf + (size_t)i * a.C;
    float lm = -INFINITY;
    for (int k = tid; k < a.C; k += AD_NT) lm = fmaxf(lm, lg[k]);
    lm = bmax(lm, red);
    float s = 0.f;
    for (int k = tid; k < a.C; k += AD_NT) s += expf(lg[k] - lm);
    s = bsum(s, red);
    const float c = 1.0f / s;
    fire = (a.delta < 1.0f) && (c >= a.delta);
    if (tid == 0 && a.tr_c) a.tr_c[tr_row] = c;
    if (fire) {
      for (int k = tid; k < a.C; k += AD_NT) a.logits[(size_t)orig * a.C + k] = lg[k];
      if (tid == 0) a.exit_block[orig] = a.b;
    }
  }

  // ----------------------------------------------------------- prune --
  if (a.isP && !fire && a.prune_rule == 1) {
    // s_t = w . z_t + beta on the merged rows (Eq. 8): one half wave per
    // token, 16-byte pieces, fixed-order half-wave sum.  The merge's row
    // writes above are visible here: same workgroup, past a barrier.
    const int hw = tid >> 5, hl = tid & 31, d4 = d >> 2;
    const float4* w4 = (const float4*)a.prune_w;
    const float pb = a.prune_b[0];
    for (int t = 1 + hw; t < T; t += AD_NT / 32) {
      if (!keepf[t]) continue;
      const float4* xr = (const float4*)(a.x + (size_t)(base + t) * d);
      float s = 0.f;
      for (int q = hl; q < d4; q += 32) {
        const float4 v = xr[q], w = w4[q];
        s = fmaf(v.x, w.x, s);
        s = fmaf(v.y, w.y, s);
        s = fmaf(v.z, w.z, s);
        s = fmaf(v.w, w.w, s);
      }
      s = half_sum(s);
      if (hl == 0) sc[t] = s + pb;
    }
    __syncthreads();
  }
  if (a.isP && !fire) {
    int ns = 0;
    for (int t = 1 + tid; t < T; t += AD_NT) ns += keepf[t];
    ns = bsum_i(ns, ired);
    const int k = (int)floor(__dmul_rn(a.tau_eff, (double)ns));
    constexpr int U = (TMAX + AD_NT - 1) / AD_NT;
    int keep_new[U];
#pragma unroll
    for (int u = 0; u < U; u++) {
      const int t = 1 + tid + u * AD_NT;
      keep_new[u] = 0;
      if (t < T && keepf[t]) {
        const float v = sc[t];
        int rank = 0;
        for (int t2 = 1; t2 < T; t2++)
          if (keepf[t2]) rank += (sc[t2] > v) || (sc[t2] == v && t2 < t);
        keep_new[u] = rank < k;
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < U; u++) {
      const int t = 1 + tid + u * AD_NT;
      if (t < T) keepf[t] = keep_new[u];
    }
    __syncthreads();
  }

  int cnt = 0;
  for (int t = tid; t < T; t += AD_NT) {
    const int kf = fire ? 0 : keepf[t];
    a.keep[base + t] = kf;
    cnt += kf;
  }
  cnt = bsum_i(cnt, ired);
  if (tid == 0) a.newlen[i] = cnt;
}

hipError_t launch_adapt(const AdaptArgs& a, hipStream_t s) {
  if (a.nlive_ub <= 0) return hipSuccess;
  if (a.n0 + 1 <= 256) {
    if (a.d % AdSize<256>::SKC != 0) return hipErrorInvalidValue;
    adapt_kernel<AdSize<256>><<<a.nlive_ub, AD_NT, 0, s>>>(a);
  } else {
    if (a.n0 + 1 > AD_TMAX || a.d % AdSize<AD_TMAX>::SKC != 0) return hipErrorInvalidValue;
    adapt_kernel<AdSize<AD_TMAX>><<<a.nlive_ub, AD_NT, 0, s>>>(a);
  }
  return hipGetLastError();
}

// --------------------------------------------------------- compaction --
// Grid: (live sample, part); every workgroup of a sample recomputes the
// sample's offsets (cheap scans) and moves one contiguous range of its rows.
constexpr int CP_PARTS = 8;
template <typename T>
__global__ __launch_bounds__(256) void compact_kernel(CompactArgs a) {
  const int i = blockIdx.x, part = blockIdx.y;
  const int nl = a.cnt->nlive;
  // Workgroup (0, 0) always publishes the next counters, also when no sample
  // is live any more (the next block must see nlive = 0, not a stale value).
  if (i >= nl && (i != 0 || part != 0)) return;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  __shared__ int ired[8];
  __shared__ int dsts[AD_TMAX];
  __shared__ int chunk_off[AD_TMAX / 64 + 1];

  int off = 0, j = 0;
  for (int t = tid; t < i; t += 256) {
    const int n = a.newlen[t];
    off += n;
    j += n > 0;
  }
  off = block_sum256_i(off, ired);
  j = block_sum256_i(j, ired);
  if (i == 0 && part == 0) {
    int tot = 0, nn = 0;
    for (int t = tid; t < nl; t += 256) {
      const int n = a.newlen[t];
      tot += n;
      nn += n > 0;
    }
    tot = block_sum256_i(tot, ired);
    nn = block_sum256_i(nn, ired);
    if (tid == 0) {
      a.cnt2->nlive = nn;
      a.cnt2->M = tot;
      a.cu2[nn] = tot;
    }
  }
  if (i >= nl || a.newlen[i] == 0) return;
  const int base = a.cu[i], Tn = a.cu[i + 1] - base;
  const int orig = a.live[i];
  if (tid == 0 && part == 0) {
    a.cu2[j] = off;
    a.live2[j] = orig;
  }
  const int nch = (Tn + 63) / 64;
  for (int c = wave; c < nch; c += 4) {
    const int t = c * 64 + lane;
    const unsigned long long msk = __ballot(t < Tn && a.keep[base + t]);
    if (lane == 0) chunk_off[c] = __popcll(msk);
  }
  __syncthreads();
  if (tid == 0) {
    int run = 0;
    for (int c = 0; c < nch; c++) {
      const int n = chunk_off[c];
      chunk_off[c] = run;
      run += n;
    }
  }
  __syncthreads();
  for (int c = wave; c < nch; c += 4) {
    const int t = c * 64 + lane;
    const bool f = t < Tn && a.keep[base + t];
    const unsigned long long msk = __ballot(f);
    const int pos = __popcll(msk & ((1ull << lane) - 1ull));
    if (t < Tn) dsts[t] = f ? chunk_off[c] + pos : -1;
  }
  __syncthreads();
  // kept rows of this part (the sample's rows split into CP_PARTS ranges):
  // one half wave per row copies it (16-byte pieces) and, when asked,
  // writes its LayerNorm for the next block
  const int per = (Tn + CP_PARTS - 1) / CP_PARTS;
  const int t0 = part * per, t1 = min(Tn, t0 + per);
  for (int t = t0 + (tid >> 5); t < t1; t += 8) {
    const int dj = dsts[t];
    if (dj < 0) continue;
    const size_t dr = (size_t)(off + dj);
    ln_row_half<T>(a.x + (size_t)(base + t) * a.d, a.d, lane & 31, a.ln_g, a.ln_b,
                   a.ln_out ? (T*)a.ln_out + dr * a.d : nullptr, a.x2 + dr * a.d);
  }
  for (int t = t0 + tid; t < t1; t += 256) {
    const int dj = dsts[t];
    if (dj < 0) continue;
    a.size2[off + dj] = a.size[base + t];
    a.origin2[off + dj] = a.origin[base + t];
    if (a.tr_ids)
      a.tr_ids[((size_t)(a.b - 1) * a.B + orig) * (a.n0 + 1) + dj] = a.origin[base + t];
  }
}

template <typename T>
hipError_t launch_compact(const CompactArgs& a, hipStream_t s) {
  if (a.nlive_ub <= 0) return hipSuccess;
  if (a.n0 + 1 > AD_TMAX || a.d % 4 != 0 || a.d > 4 * 32 * LN_MAXV) return hipErrorInvalidValue;
  compact_kernel<T><<<dim3(a.nlive_ub, CP_PARTS), 256, 0, s>>>(a);
  return hipGetLastError();
}
template hipError_t launch_compact<float>(const CompactArgs&, hipStream_t);
template hipError_t launch_compact<bf16_t>(const CompactArgs&, hipStream_t);

}  // namespace fusion
