// Per-sample adaptive steps after a block (Algorithm 1, Sec. III-B..E):
//   merge router and count (Eq. 4-5), bipartite soft matching with
//   size-weighted merging (Sec. III-C), exit check on the CLS head
//   (Eq. 6-7), CLS-attention top-k pruning of continuing samples (Eq. 8),
// followed by a separate compaction kernel that re-packs the surviving
// samples and tokens (exclusive scans over new lengths and keep flags).
// The fp32 rows of x never move: a token keeps its physical row (a merge
// updates the destination row in place) and the compaction re-packs the row
// map, the sizes and the origin ids.
//
// One 512-thread workgroup per live sample (the compaction uses 256).  No
// float atomics: every reduction has a fixed order, so results do not depend
// on scheduling or on the rest of the batch.
#include "kernels.h"

namespace fusion {

constexpr int AD_TMAX = 640;  // tokens per sample (CLS included), largest size class
constexpr int AD_NT = 512;    // threads per workgroup (8 waves)

// Size classes of the per-sample kernel: TMAX tokens (CLS included), so
// |A| = ceil(N/2) and |B| = floor(N/2) are at most TMAX/2.  The smallest
// class (T <= 128, picked from the host's token bound of the block) stages
// 64 features per chunk: its chunk loop is latency-bound, and half the
// chunks halve the barriers.
template <int TMAX_, int WC_ = (TMAX_ <= 128 ? 4 : TMAX_ <= 256 ? 2 : 4)> struct AdSize {
  static constexpr int TMAX = TMAX_;
  static constexpr int AMAX = TMAX_ / 2;
  static constexpr int BMAX = TMAX_ / 2;
  static constexpr int SKC = TMAX_ <= 128 ? 64 : 32;  // features per chunk (MFMA K steps of 32)
  // LDS row of a staged chunk (bf16): 32-feature chunks are unpadded 64-byte
  // rows with their four 16-byte pieces XOR-permuted by (row / 4) % 4 (the
  // 16-byte operand reads of 16 consecutive rows then hit disjoint banks);
  // 64-feature chunks are padded to 144-byte rows
  static constexpr bool SWZ = SKC == 32;
  static constexpr int SKP = SWZ ? SKC : SKC + 8;
  // similarity wave layout: WC column groups of B tiles, AD_NT / 64 / WC
  // groups of 32 A rows; SAG A rows per pass
  static constexpr int WC = WC_;
  static constexpr int SAG = 32 * (AD_NT / 64 / WC);
  static constexpr int NBT = BMAX / 16;        // B tiles of 16 rows
  static constexpr int NBW = NBT / WC;         // B tiles per wave
  static constexpr int BG = TMAX_ <= 128 ? 1 : TMAX_ <= 256 ? 4 : 5;  // B tiles per MFMA group
  static constexpr int SPT = ((SAG + BMAX) * (SKC / 4) + AD_NT - 1) / AD_NT;  // slots / thread
};

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
static_assert(AdSize<AD_TMAX>::AMAX == AD_SIM_STRIDE, "similarity workspace stride");

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

// Lanes that share one element's rank count when n elements are ranked by
// the workgroup: the largest power of two (at most 16) with n * P <= AD_NT.
__device__ __forceinline__ int rank_lanes(int n) {
  int P = 1;
  while (P < 16 && n * (2 * P) <= AD_NT) P *= 2;
  return P;
}

// Order-preserving key of a float: for a, b not NaN, a < b iff
// order_key(a) < order_key(b), and a == b iff the keys are equal (-0 and +0
// share the key of +0).
__device__ __forceinline__ unsigned order_key(float f) {
  const unsigned u = f == 0.f ? 0u : __float_as_uint(f);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

// Top-c selection over the workgroup, E (1 or 2) elements per thread:
// e = tid (key k0, taking part if ok0) and e = tid + AD_NT (k1, ok1).  An
// element is chosen iff it takes part and fewer than c participating
// elements precede it, a larger key or an equal key at a lower e coming
// first: the rank rule of the merge and prune selections (ties to the lower
// slot), without the all-pairs comparisons.  The c-th largest key is found
// two bits at a time from the top: per round one workgroup count of the
// candidates whose next two bits are >= 1, >= 2 and 3 (a ballot per wave
// and count, the wave counts in LDS slots used alternately, so one barrier
// per round); then the elements equal to it are taken in ascending e until
// c are chosen.  cnt: 6 * AD_NT / 64 ints of LDS; the caller synchronises
// before reusing them.
template <int E>
__device__ __forceinline__ void block_top(unsigned k0, bool ok0, unsigned k1, bool ok1, int c,
                                          bool& ch0, bool& ch1, int* cnt) {
  constexpr int NW = AD_NT / 64;
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  if (E < 2) ok1 = false;
  ch0 = ch1 = false;
  if (c <= 0) return;
  unsigned prefix = 0, mask = 0;
  int need = c, slot = 1;
  for (int bit = 30; bit >= 0; bit -= 2) {
    const bool m0 = ok0 && (k0 & mask) == prefix, m1 = ok1 && (k1 & mask) == prefix;
    const unsigned g0 = (k0 >> bit) & 3u, g1 = (k1 >> bit) & 3u;
    int n[3];
#pragma unroll
    for (int q = 0; q < 3; q++) {
      n[q] = __popcll(__ballot(m0 && g0 >= (unsigned)(q + 1)));
      if (E > 1) n[q] += __popcll(__ballot(m1 && g1 >= (unsigned)(q + 1)));
    }
    if (lane == 0) {
#pragma unroll
      for (int q = 0; q < 3; q++) cnt[(slot * 3 + q) * NW + wave] = n[q];
    }
    __syncthreads();
    int ge[3] = {0, 0, 0};  // candidates whose next two bits are >= 1, >= 2, == 3
#pragma unroll
    for (int q = 0; q < 3; q++)
#pragma unroll
      for (int w = 0; w < NW; w++) ge[q] += cnt[(slot * 3 + q) * NW + w];
    slot ^= 1;
    unsigned g;
    if (ge[2] >= need) {
      g = 3u;
    } else if (ge[1] >= need) {
      g = 2u;
      need -= ge[2];
    } else if (ge[0] >= need) {
      g = 1u;
      need -= ge[1];
    } else {
      g = 0u;
      need -= ge[0];
    }
    prefix |= g << bit;
    mask |= 3u << bit;
  }
  // the elements equal to the c-th key, in ascending e: all of the first
  // half (e < AD_NT) come before the second
  const bool eq0 = ok0 && k0 == prefix, eq1 = ok1 && k1 == prefix;
  const unsigned long long b0 = __ballot(eq0), b1 = E > 1 ? __ballot(eq1) : 0ull;
  __syncthreads();
  if (lane == 0) {
    cnt[wave] = __popcll(b0);
    cnt[NW + wave] = __popcll(b1);
  }
  __syncthreads();
  int before0 = 0, before1 = 0, tot0 = 0;
#pragma unroll
  for (int w = 0; w < NW; w++) {
    tot0 += cnt[w];
    before0 += w < wave ? cnt[w] : 0;
    before1 += w < wave ? cnt[NW + w] : 0;
  }
  const unsigned long long lt = (1ull << lane) - 1ull;
  const int r0 = before0 + __popcll(b0 & lt);
  const int r1 = tot0 + before1 + __popcll(b1 & lt);
  ch0 = ok0 && (k0 > prefix || (eq0 && r0 < need));
  ch1 = ok1 && (k1 > prefix || (eq1 && r1 < need));
}

// Candidates above which block_top replaces the all-pairs rank count (its
// rounds cost about as much as 256 rank comparisons per thread).
constexpr int SEL_RADIX_MIN = 256;

// Cosine similarities of the A tokens (even patch slots) with the B tokens
// (odd slots) of one sample, and the best B for every A.
//
// One pass over the features in chunks of SKC, double-buffered in LDS.
// The token rows are read from x through prow (the sample's physical row of
// each token slot).  Every thread owns a fixed set of (row, 4-feature)
// slots: the A rows of the pass first, then the B rows (clamped to the last
// real row, so
// the loads need no branch; padding rows only feed outputs that are never
// read).  The loads run two chunks ahead in two register sets.  A chunk's
// values are split into bf16 hi + lo (hi = RNE(v), lo = RNE(v - hi)), with
// the row's sum of squares accumulated on the way, and written to the LDS
// buffer that the MFMAs of the current chunk do not read: one barrier per
// chunk.  The dot products take hi.hi' + hi.lo' + lo.hi' on
// v_mfma_f32_16x16x32_bf16 with fp32 accumulation (absolute error of a
// cosine <= ~1.2e-5, the dropped lo.lo' term included), per output in
// feature order, the three terms in that order within each 32 features.
// The B fragment is the MFMA's row operand, so lane l of a 16 x 16 output
// tile holds S[b = 4 (l / 16) + j][a = l % 16] (j = 0..3): the candidates
// of one A token sit in 4 lanes x 4 registers per B tile.  Wave w owns A
// rows 32 (w / WC) .. +31 of the pass against B tiles NBW (w % WC) .. +NBW-1.
// Cosines are dot * (1 / n_a) * (1 / n_b) with the clamped norms
// max(||x||, 1e-12).  The argmax over B (ties to the lowest B index, NaN
// never wins) runs in-lane, then across the 4 lanes of a token with the
// lane-swap instructions, then over the WC wave groups in B order through
// LDS (pbv, pbi: WC SAG entries each).  rn holds the reciprocal norms:
// A rows of the pass at [0, SAG), B rows at [SAG, SAG + BMAX).  Passes of SAG
// A rows run from A row ag_first, at most n_pass of them; bestsim / best may
// point to LDS or to global memory (indexed by A row).
template <class Z>
__device__ void similarity_argmax(const float* __restrict__ x, const int* prow, int d,
                                  int nA, int nB, float* rn, float* bestsim,
                                  int* best, bf16_t* Ahi, bf16_t* Alo,
                                  bf16_t* Bhi, bf16_t* Blo, float* pbv, int* pbi,
                                  int ag_first = 0, int n_pass = 1 << 30) {
  constexpr int SKC = Z::SKC, SKP = Z::SKP, SPT = Z::SPT, NBW = Z::NBW, BG = Z::BG;
  constexpr int SAG = Z::SAG, WC = Z::WC, BMAX = Z::BMAX;
  constexpr int Q = SKC / 4;  // 16-byte slots per row and chunk
  static_assert(SKC % 32 == 0, "whole MFMA K steps per chunk");
  static_assert(SPT * AD_NT == (SAG + BMAX) * Q, "slots must tile the staged rows exactly");
  static_assert(NBW % BG == 0 && NBW * WC == Z::NBT, "wave layout: B tiles split evenly");
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int g = lane >> 4, c = lane & 15;
  const int wr = wave / WC, wc = wave % WC;
  const int nbt = (nB + 15) >> 4, nck = d / SKC;
  for (int ag = ag_first, pass = 0; ag < nA && pass < n_pass; ag += SAG, pass++) {
    const float* xs = x;
    uint32_t soff[SPT];  // slot offsets into x, in floats (physical row * d + feature)
    bool sval[SPT];
    float ss[SPT];
#pragma unroll
    for (int w = 0; w < SPT; w++) {
      const int u = tid + w * AD_NT;
      const int r = u / Q, q = (u % Q) * 4;
      if (r < SAG) {
        sval[w] = ag + r < nA;
        soff[w] = (uint32_t)prow[1 + 2 * min(ag + r, nA - 1)] * d + q;
      } else {
        sval[w] = r - SAG < nB;
        soff[w] = (uint32_t)prow[2 + 2 * min(r - SAG, nB - 1)] * d + q;
      }
      ss[w] = 0.f;
    }
    auto load = [&](float4(&cx)[SPT], int kc) {
#pragma unroll
      for (int w = 0; w < SPT; w++) cx[w] = *(const float4*)(xs + soff[w] + kc * SKC);
    };
    // split chunk values into hi / lo and write them to LDS buffer `buf`
    auto stage = [&](const float4(&cx)[SPT], int buf) {
#pragma unroll
      for (int w = 0; w < SPT; w++) {
        const float4 e = cx[w];
        ss[w] = fmaf(e.x, e.x, ss[w]);
        ss[w] = fmaf(e.y, e.y, ss[w]);
        ss[w] = fmaf(e.z, e.z, ss[w]);
        ss[w] = fmaf(e.w, e.w, ss[w]);
        const uint32_t h01 = pack_bf16x2(e.x, e.y), h23 = pack_bf16x2(e.z, e.w);
        const uint2 hv = make_uint2(h01, h23);
        const uint2 lv = make_uint2(pack_bf16x2(e.x - __uint_as_float(h01 << 16),
                                                e.y - __uint_as_float(h01 & 0xFFFF0000u)),
                                    pack_bf16x2(e.z - __uint_as_float(h23 << 16),
                                                e.w - __uint_as_float(h23 & 0xFFFF0000u)));
        const int u = tid + w * AD_NT;
        const int r = u / Q, q = (u % Q) * 4;
        bf16_t* H = r < SAG ? Ahi + (buf * SAG + r) * SKP : Bhi + (buf * BMAX + r - SAG) * SKP;
        bf16_t* Lo = r < SAG ? Alo + (buf * SAG + r) * SKP : Blo + (buf * BMAX + r - SAG) * SKP;
        // (SAG and BMAX are multiples of 16, so r % 16 is the LDS row's)
        const int qs = Z::SWZ ? ((((q >> 3) ^ (r >> 2)) & 3) << 3) | (q & 4) : q;
        *(uint2*)(H + qs) = hv;
        *(uint2*)(Lo + qs) = lv;
      }
    };
    f32x4_t acc[2][NBW];
#pragma unroll
    for (int i = 0; i < 2; i++)
#pragma unroll
      for (int t = 0; t < NBW; t++) acc[i][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};
    // wave-uniform: does this wave's block hold any real (A, B) pair
    const bool act = ag + 32 * wr < nA && wc * NBW < nbt;
    auto mfma = [&](int buf) {
      if (!act) return;
      // column of this lane's 16-byte piece (rows r with r % 16 == c)
      const int gs = Z::SWZ ? ((g ^ (c >> 2)) << 3) : 8 * g;
#pragma unroll
      for (int kk = 0; kk < SKC / 32; kk++) {
        bf16x8_t ah[2], al[2];
#pragma unroll
        for (int i = 0; i < 2; i++) {
          const int row = buf * SAG + 32 * wr + 16 * i + c;
          ah[i] = *(const bf16x8_t*)(Ahi + row * SKP + 32 * kk + gs);
          al[i] = *(const bf16x8_t*)(Alo + row * SKP + 32 * kk + gs);
        }
#pragma unroll
        for (int t0 = 0; t0 < NBW; t0 += BG) {
          bf16x8_t bh[BG], bl[BG];
#pragma unroll
          for (int j = 0; j < BG; j++) {
            const int row = buf * BMAX + (wc * NBW + t0 + j) * 16 + c;
            bh[j] = *(const bf16x8_t*)(Bhi + row * SKP + 32 * kk + gs);
            bl[j] = *(const bf16x8_t*)(Blo + row * SKP + 32 * kk + gs);
          }
#pragma unroll
          for (int j = 0; j < BG; j++)
#pragma unroll
            for (int i = 0; i < 2; i++)
              acc[i][t0 + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[j], ah[i], acc[i][t0 + j], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < BG; j++)
#pragma unroll
            for (int i = 0; i < 2; i++)
              acc[i][t0 + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bl[j], ah[i], acc[i][t0 + j], 0, 0, 0);
#pragma unroll
          for (int j = 0; j < BG; j++)
#pragma unroll
            for (int i = 0; i < 2; i++)
              acc[i][t0 + j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(bh[j], al[i], acc[i][t0 + j], 0, 0, 0);
        }
      }
    };
    // chunk kc: MFMAs on buffer kc & 1; chunk kc + 1 (in registers `nx`)
    // staged into the other buffer; chunk kc + 3 loaded into `nx`
    float4 r0[SPT], r1[SPT];
    auto step = [&](int kc, float4(&nx)[SPT]) {
      mfma(kc & 1);
      if (kc + 1 < nck) stage(nx, (kc + 1) & 1);
      if (kc + 3 < nck) load(nx, kc + 3);
      __syncthreads();
    };
    load(r0, 0);
    if (nck > 1) load(r1, 1);
    stage(r0, 0);
    if (nck > 2) load(r0, 2);
    __syncthreads();
    for (int kc = 0; kc < nck; kc += 2) {
      step(kc, r1);
      if (kc + 1 < nck) step(kc + 1, r0);
    }
    // reciprocal row norms: the Q threads of a row are adjacent lanes
#pragma unroll
    for (int w = 0; w < SPT; w++) {
      float v = ss[w];
#pragma unroll
      for (int o = 1; o < Q; o <<= 1) v += __shfl_xor(v, o, 64);
      const int u = tid + w * AD_NT;
      if (sval[w] && (u % Q) == 0) rn[u / Q] = 1.0f / fmaxf(sqrtf(v), 1e-12f);
    }
    __syncthreads();
    // best B per A over this wave's tiles; rows and columns past nA / nB
    // read clamped or stale norms and are masked
#pragma unroll
    for (int i = 0; i < 2; i++) {
      const int ar = 32 * wr + 16 * i + c;  // A row within the pass
      const float ra = rn[min(ar, max(nA - ag, 1) - 1)];
      float bv = -INFINITY;
      int bi = 0x7fffffff;
#pragma unroll
      for (int t = 0; t < NBW; t++) {
        const int b0 = (wc * NBW + t) * 16 + 4 * g;
        const float4 rb = *(const float4*)(rn + SAG + b0);
        const float rbj[4] = {rb.x, rb.y, rb.z, rb.w};
#pragma unroll
        for (int j = 0; j < 4; j++) {
          const float v = (acc[i][t][j] * ra) * rbj[j];
          const bool take = act && b0 + j < nB && v > bv;
          bv = take ? v : bv;
          bi = take ? b0 + j : bi;
        }
      }
      // combine the 4 lanes of the token (lanes c, c + 16, c + 32, c + 48):
      // each swap yields the lane's own pair and its partner's
      {
        const auto v16 = __builtin_amdgcn_permlane16_swap(__float_as_uint(bv), __float_as_uint(bv), false, false);
        const auto i16 = __builtin_amdgcn_permlane16_swap((unsigned)bi, (unsigned)bi, false, false);
        const float v0 = __uint_as_float(v16[0]), v1 = __uint_as_float(v16[1]);
        const int i0 = (int)i16[0], i1 = (int)i16[1];
        const bool t1 = v1 > v0 || (v1 == v0 && i1 < i0);
        bv = t1 ? v1 : v0;
        bi = t1 ? i1 : i0;
      }
      {
        const auto v32 = __builtin_amdgcn_permlane32_swap(__float_as_uint(bv), __float_as_uint(bv), false, false);
        const auto i32 = __builtin_amdgcn_permlane32_swap((unsigned)bi, (unsigned)bi, false, false);
        const float v0 = __uint_as_float(v32[0]), v1 = __uint_as_float(v32[1]);
        const int i0 = (int)i32[0], i1 = (int)i32[1];
        const bool t1 = v1 > v0 || (v1 == v0 && i1 < i0);
        bv = t1 ? v1 : v0;
        bi = t1 ? i1 : i0;
      }
      if (g == 0) {
        pbv[wc * SAG + ar] = bv;
        pbi[wc * SAG + ar] = bi;
      }
    }
    __syncthreads();
    // partial results in B order: a later group wins only on a larger value
    for (int e = tid; e < SAG && ag + e < nA; e += AD_NT) {
      float v0 = pbv[e];
      int i0 = pbi[e];
#pragma unroll
      for (int w = 1; w < WC; w++) {
        const float v1 = pbv[w * SAG + e];
        const int i1 = pbi[w * SAG + e];
        if (v1 > v0 || (v1 == v0 && i1 < i0)) {
          v0 = v1;
          i0 = i1;
        }
      }
      bestsim[ag + e] = v0;
      best[ag + e] = i0 < nB ? i0 : 0;  // i0 >= nB only with non-finite x
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

  constexpr int TMAX = Z::TMAX, AMAX = Z::AMAX, BMAX = Z::BMAX, SKP = Z::SKP, SAG = Z::SAG;
  static_assert(AMAX <= AD_NT && TMAX - 1 <= 2 * AD_NT, "block_top covers every candidate");
  // the host's token bound selects the size class and is exact; a sample
  // beyond it (never produced by the library itself) is dropped rather than
  // overrunning the per-token LDS arrays
  if (T > TMAX || T < 1) {
    if (tid == 0) a.newlen[i] = 0;
    return;
  }
  __shared__ float sc[TMAX];
  __shared__ float szs[TMAX];
  __shared__ int prow[TMAX];  // physical row of x for each of the sample's tokens
  __shared__ int keepf[TMAX];
  __shared__ int knew[TMAX];
  __shared__ __attribute__((aligned(16))) float rn[TMAX];  // reciprocal norms
  __shared__ float bestsim[AMAX];
  __shared__ int best[AMAX];
  __shared__ int chosen[AMAX];
  __shared__ int clist[AMAX];
  __shared__ int cdst[AMAX];
  __shared__ int glead[AMAX];
  __shared__ int srt[AMAX];
  __shared__ float tmpf[AMAX];
  __shared__ float tmps[AMAX];
  // similarity operands, two buffers each
  __shared__ __attribute__((aligned(16))) bf16_t Ahi[2 * SAG * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Alo[2 * SAG * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Bhi[2 * BMAX * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Blo[2 * BMAX * SKP];
  __shared__ float pbv[Z::WC * SAG];
  __shared__ int pbi[Z::WC * SAG];
  __shared__ float red[16];
  __shared__ int ired[16];
  __shared__ int selc[6 * AD_NT / 64];  // block_top's counts

  // CLS-attention scores are gathered here and follow the merge; learned
  // scores are computed after the merge from the merged hidden states
  const bool attnP = a.isP && a.prune_rule == 0;
  for (int t = tid; t < T; t += AD_NT) {
    keepf[t] = 1;
    szs[t] = a.size[base + t];
    prow[t] = a.rmap[base + t];
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
  if (a.isM && a.r_fixed) {
    r = min(max(a.r_fixed[i], 0), N / 2);
    if (tid == 0 && a.tr_r) a.tr_r[tr_row] = r;
  } else if (a.isM) {
    float z = 0.f;
    const float* xc = a.x + (size_t)prow[0] * d;
    for (int k = tid; k < d; k += AD_NT) z = fmaf(a.router_w[k], xc[k], z);
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
    if (a.sim_v) {
      // best matches computed by similarity_kernel, one workgroup per pass
      for (int e = tid; e < nA; e += AD_NT) {
        bestsim[e] = a.sim_v[(size_t)i * AMAX + e];
        best[e] = a.sim_i[(size_t)i * AMAX + e];
      }
      __syncthreads();
    } else {
      similarity_argmax<Z>(a.x, prow, d, nA, nB, rn, bestsim, best, Ahi, Alo, Bhi, Blo, pbv,
                           pbi);
    }
    // top-r of A by best similarity, ties to the lower A slot: a radix
    // selection for many candidates (nA <= AD_NT), else the rank count with
    // P adjacent lanes splitting the comparisons of one element
    if (nA > SEL_RADIX_MIN) {
      const bool ok = tid < nA;
      bool ch, unused;
      block_top<1>(order_key(ok ? bestsim[tid] : 0.f), ok, 0u, false, r, ch, unused, selc);
      if (ok) chosen[tid] = ch;
    } else {
      const int P = rank_lanes(nA), p = tid % P;
      for (int e0 = 0; e0 < nA; e0 += AD_NT / P) {
        const int aa = e0 + tid / P;
        int rank = 0;
        if (aa < nA) {
          const float v = bestsim[aa];
          for (int a2 = p; a2 < nA; a2 += P) {
            const float v2 = bestsim[a2];
            rank += (v2 > v) || (v2 == v && a2 < aa);
          }
        }
        for (int o = 1; o < P; o <<= 1) rank += __shfl_xor(rank, o, 64);
        if (aa < nA && p == 0) chosen[aa] = rank < r;
      }
    }
    __syncthreads();
    // chosen sources in ascending A slot: clist[0 .. r)
    block_compact(tid < nA && chosen[tid], tid, clist, ired);
    // destination of each, and the sources sorted by (destination, A slot):
    // srt[0 .. r) lists the positions q in clist; the sources of one
    // destination form a group, contiguous in srt and in ascending A slot.
    // Groups are merged independently.
    for (int q = tid; q < r; q += AD_NT) cdst[q] = best[clist[q]];
    __syncthreads();
    {
      const int P = rank_lanes(r), p = tid % P;
      for (int e0 = 0; e0 < r; e0 += AD_NT / P) {
        const int q = e0 + tid / P;
        int rank = 0;
        if (q < r) {
          const int key = cdst[q];
          for (int q2 = p; q2 < r; q2 += P) {
            const int k2 = cdst[q2];
            rank += (k2 < key) || (k2 == key && q2 < q);
          }
        }
        for (int o = 1; o < P; o <<= 1) rank += __shfl_xor(rank, o, 64);
        if (q < r && p == 0) srt[rank] = q;
      }
    }
    __syncthreads();
    const bool start = tid < r && (tid == 0 || cdst[srt[tid]] != cdst[srt[tid - 1]]);
    const int ng = block_compact(start, tid, glead, ired);  // glead[k]: first position of group k
    // size-weighted merge into each receiving destination (16-byte pieces);
    // the destination row and the group's first source are loaded together
    const int d4 = d / 4;
    float4* x4 = (float4*)a.x;
    for (int idx = tid; idx < ng * d4; idx += AD_NT) {
      const int k = idx / d4, f = idx - k * d4;
      const int p0 = glead[k], p1 = k + 1 < ng ? glead[k + 1] : r;
      const int bb = cdst[srt[p0]], a0 = clist[srt[p0]];
      const size_t rowb = (size_t)prow[2 + 2 * bb];
      const float4 xb = x4[rowb * d4 + f];
      const float4 xa0 = x4[(size_t)prow[1 + 2 * a0] * d4 + f];
      const float sb = szs[2 + 2 * bb], sa0 = szs[1 + 2 * a0];
      float4 num = make_float4(sb * xb.x, sb * xb.y, sb * xb.z, sb * xb.w);
      num.x = num.x + sa0 * xa0.x;
      num.y = num.y + sa0 * xa0.y;
      num.z = num.z + sa0 * xa0.z;
      num.w = num.w + sa0 * xa0.w;
      float den = sb + sa0;
      for (int pp = p0 + 1; pp < p1; pp++) {
        const int aa = clist[srt[pp]];
        const float sa = szs[1 + 2 * aa];
        const float4 xa = x4[(size_t)prow[1 + 2 * aa] * d4 + f];
        num.x = num.x + sa * xa.x;
        num.y = num.y + sa * xa.y;
        num.z = num.z + sa * xa.z;
        num.w = num.w + sa * xa.w;
        den = den + sa;
      }
      x4[rowb * d4 + f] = make_float4(num.x / den, num.y / den, num.z / den, num.w / den);
    }
    for (int k = tid; k < ng; k += AD_NT) {
      const int p0 = glead[k], p1 = k + 1 < ng ? glead[k + 1] : r;
      const int bb = cdst[srt[p0]];
      float den = szs[2 + 2 * bb];
      float s2 = attnP ? sc[2 + 2 * bb] : 0.f;
      for (int pp = p0; pp < p1; pp++) {
        const int aa = clist[srt[pp]];
        den = den + szs[1 + 2 * aa];
        if (attnP) s2 = s2 + sc[1 + 2 * aa];
      }
      tmpf[k] = den;
      tmps[k] = s2;
    }
    __syncthreads();
    for (int k = tid; k < ng; k += AD_NT) {
      const int bb = cdst[srt[glead[k]]];
      a.size[base + 2 + 2 * bb] = tmpf[k];
      if (attnP) sc[2 + 2 * bb] = tmps[k];
    }
    for (int q = tid; q < r; q += AD_NT) {
      const int aa = clist[q];
      keepf[1 + 2 * aa] = 0;
      if (a.tr_merge) {
        const int so = a.origin[base + 1 + 2 * aa];
        if (so >= 0 && so <= a.n0)
          a.tr_merge[tr_row * (a.n0 + 1) + so] = a.origin[base + 2 + 2 * best[aa]];
      }
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
      const float4* xr = (const float4*)(a.x + (size_t)prow[t] * d);
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
    // top-k of the kept patch tokens by score, ties to the lower slot: a
    // radix selection for many candidates (patch token t = 1 + e,
    // T - 1 <= 2 AD_NT), else the rank count with P adjacent lanes
    // splitting the comparisons of one token
    if (T - 1 > SEL_RADIX_MIN) {
      const int t0 = 1 + tid, t1 = 1 + AD_NT + tid;
      const bool ok0 = t0 < T && keepf[t0], ok1 = t1 < T && keepf[t1];
      bool ch0, ch1;
      block_top<2>(order_key(ok0 ? sc[t0] : 0.f), ok0, order_key(ok1 ? sc[t1] : 0.f), ok1, k,
                   ch0, ch1, selc);
      if (t0 < T) knew[t0] = ch0;
      if (t1 < T) knew[t1] = ch1;
    } else {
      const int P = rank_lanes(T - 1), p = tid % P;
      for (int e0 = 0; e0 < T - 1; e0 += AD_NT / P) {
        const int t = 1 + e0 + tid / P;
        const bool act = t < T && keepf[t];
        int rank = 0;
        if (act) {
          const float v = sc[t];
          for (int t2 = 1 + p; t2 < T; t2 += P) {
            const float v2 = sc[t2];
            rank += keepf[t2] & ((v2 > v) | (v2 == v && t2 < t));
          }
        }
        for (int o = 1; o < P; o <<= 1) rank += __shfl_xor(rank, o, 64);
        if (t < T && p == 0) knew[t] = act && rank < k;
      }
    }
    __syncthreads();
    for (int t = 1 + tid; t < T; t += AD_NT) keepf[t] = knew[t];
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

// Best matches of the merge step for long samples, one workgroup per (live
// sample, pass of SAG A rows): the same passes similarity_argmax makes one
// after the other inside adapt_kernel, spread over workgroups so that a
// small batch of long samples fills the GPU.  Results go to a.sim_v /
// a.sim_i ([live sample][AMAX]); adapt_kernel reads them instead.
template <class Z>
__global__ __launch_bounds__(AD_NT) void similarity_kernel(AdaptArgs a) {
  const int i = blockIdx.x, pass = blockIdx.y;
  if (i >= a.cnt->nlive) return;
  const int base = a.cu[i], T = a.cu[i + 1] - base, N = T - 1;
  if (T > Z::TMAX || T < 1) return;
  const int nA = (N + 1) / 2, nB = N / 2;
  if (nB < 1 || pass * Z::SAG >= nA) return;
  constexpr int TMAX = Z::TMAX, BMAX = Z::BMAX, SKP = Z::SKP, SAG = Z::SAG;
  __shared__ int prow[TMAX];
  __shared__ __attribute__((aligned(16))) float rn[TMAX];
  __shared__ __attribute__((aligned(16))) bf16_t Ahi[2 * SAG * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Alo[2 * SAG * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Bhi[2 * BMAX * SKP];
  __shared__ __attribute__((aligned(16))) bf16_t Blo[2 * BMAX * SKP];
  __shared__ float pbv[Z::WC * SAG];
  __shared__ int pbi[Z::WC * SAG];
  for (int t = threadIdx.x; t < T; t += AD_NT) prow[t] = a.rmap[base + t];
  __syncthreads();
  similarity_argmax<Z>(a.x, prow, a.d, nA, nB, rn, a.sim_v + (size_t)i * Z::AMAX,
                       a.sim_i + (size_t)i * Z::AMAX, Ahi, Alo, Bhi, Blo, pbv, pbi,
                       pass * SAG, 1);
}

hipError_t launch_adapt(const AdaptArgs& a, hipStream_t s) {
  if (a.nlive_ub <= 0) return hipSuccess;
  AdaptArgs one = a;  // single-pass classes: the adapt kernel computes the matches itself
  one.sim_v = nullptr;
  one.sim_i = nullptr;
  if (a.T_ub <= 128 && a.d % AdSize<128>::SKC == 0) {
    adapt_kernel<AdSize<128>><<<a.nlive_ub, AD_NT, 0, s>>>(one);
  } else if (a.T_ub <= 256) {
    if (a.d % AdSize<256>::SKC != 0) return hipErrorInvalidValue;
    adapt_kernel<AdSize<256>><<<a.nlive_ub, AD_NT, 0, s>>>(one);
  } else {
    typedef AdSize<AD_TMAX> Z;
    // the split similarity: passes of 128 A rows (8 waves as 4 groups of 32
    // A rows x 2 column groups), so that each sample's B rows are read
    // ceil(nA / 128) times
    typedef AdSize<AD_TMAX, 2> ZS;
    static_assert(ZS::AMAX == Z::AMAX, "one match stride for both kernels");
    if (a.T_ub > AD_TMAX || a.d % Z::SKC != 0) return hipErrorInvalidValue;
    AdaptArgs b = a;
    if (a.isM && a.sim_v && a.sim_i) {
      // several passes of A rows: one workgroup each
      const int passes = (a.T_ub / 2 + ZS::SAG - 1) / ZS::SAG;
      similarity_kernel<ZS><<<dim3(a.nlive_ub, passes), AD_NT, 0, s>>>(a);
    } else {
      b.sim_v = nullptr;
      b.sim_i = nullptr;
    }
    adapt_kernel<Z><<<a.nlive_ub, AD_NT, 0, s>>>(b);
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
  if (Tn > AD_TMAX) return;  // never kept by the adapt kernel (newlen 0)
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
  // when asked, one half wave per row writes its LayerNorm for the next
  // block (16-byte pieces); the row itself stays where it is, only its
  // physical row id, size and origin move to the packed slot
  const int per = (Tn + CP_PARTS - 1) / CP_PARTS;
  const int t0 = part * per, t1 = min(Tn, t0 + per);
  if (a.ln_out) {
    for (int t = t0 + (tid >> 5); t < t1; t += 8) {
      const int dj = dsts[t];
      if (dj < 0) continue;
      const size_t dr = (size_t)(off + dj);
      ln_row_half<T>(a.x + (size_t)a.rmap[base + t] * a.d, a.d, lane & 31, a.ln_g, a.ln_b,
                     (T*)a.ln_out + dr * a.d, nullptr);
    }
  }
  for (int t = t0 + tid; t < t1; t += 256) {
    const int dj = dsts[t];
    if (dj < 0) continue;
    a.rmap2[off + dj] = a.rmap[base + t];
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
