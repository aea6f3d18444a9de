// Per-sample adaptive steps after a block (Algorithm 1, Sec. III-B..E):
//   merge router and count (Eq. 4-5), bipartite soft matching with
//   size-weighted merging (Sec. III-C), exit check on the CLS head
//   (Eq. 6-7), CLS-attention top-k pruning of continuing samples (Eq. 8),
// followed by a separate compaction kernel that re-packs the surviving
// samples and tokens (exclusive scans over new lengths and keep flags).
//
// One 256-thread workgroup per live sample.  No float atomics: every
// reduction has a fixed order, so results do not depend on scheduling or on
// the rest of the batch.
#include "kernels.h"

namespace fusion {

constexpr int AD_TMAX = 640;  // tokens per sample (CLS included)
constexpr int AD_AMAX = 320;  // |A| = ceil(N/2)
constexpr int KC = 16;        // feature chunk of the similarity tiles
constexpr int AG = 64;        // A rows per similarity pass
constexpr int BG = 128;       // B rows per similarity pass

__device__ __forceinline__ int merge_count(float m, double rho, int r_b, int N) {
  // r = clamp(floor(((2 rho) m) r_b + 1/2), 0, floor(N/2)), every step an
  // individually rounded IEEE double operation.
  const double t = __dadd_rn(__dmul_rn(__dmul_rn(__dmul_rn(2.0, rho), (double)m),
                                       (double)r_b), 0.5);
  int r = (int)floor(t);
  if (r < 0) r = 0;
  if (r > N / 2) r = N / 2;
  return r;
}

__global__ __launch_bounds__(256) void adapt_kernel(AdaptArgs a) {
  const int i = blockIdx.x;
  if (i >= a.cnt->nlive) return;
  const int tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
  const int base = a.cu[i], T = a.cu[i + 1] - base, N = T - 1;
  const int orig = a.live[i];
  const int d = a.d;
  const size_t tr_row = (size_t)(a.b - 1) * a.B + orig;

  __shared__ float sc[AD_TMAX];
  __shared__ int keepf[AD_TMAX];
  __shared__ float nrm[AD_TMAX];
  __shared__ float bestsim[AD_AMAX];
  __shared__ int best[AD_AMAX];
  __shared__ int chosen[AD_AMAX];
  __shared__ int clist[AD_AMAX];
  __shared__ float tmpf[AD_AMAX];
  __shared__ float tmps[AD_AMAX];
  __shared__ float xa[AG][KC + 1];
  __shared__ float xb[BG][KC + 1];
  __shared__ float rbv[16][AG];
  __shared__ int rbi[16][AG];
  __shared__ float red[8];
  __shared__ int ired[8];

  for (int t = tid; t < T; t += 256) keepf[t] = 1;
  if (a.isP) {
    for (int t = tid; t < T; t += 256) {
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
    for (int k = tid; k < d; k += 256) z = fmaf(a.router_w[k], a.x[(size_t)base * d + k], z);
    z = block_sum256(z, red) + a.router_b[0];
    const float m = 1.0f / (1.0f + expf(-z));
    r = merge_count(m, a.rho, a.r_b, N);
    if (tid == 0) {
      if (a.tr_r) a.tr_r[tr_row] = r;
      if (a.tr_m) a.tr_m[tr_row] = m;
    }
  }
  const int nA = (N + 1) / 2, nB = N / 2;
  if (r > 0) {
    // clamped L2 norms of the patch tokens
    for (int j = wave; j < N; j += 4) {
      const float* xr = a.x + (size_t)(base + 1 + j) * d;
      float ss = 0.f;
      for (int k = lane; k < d; k += 64) ss = fmaf(xr[k], xr[k], ss);
      ss = wave_sum(ss);
      if (lane == 0) nrm[j] = fmaxf(sqrtf(ss), 1e-12f);
    }
    __syncthreads();
    // cosine similarities A x B in passes of AG x BG; running argmax per A
    const int ta = tid & 15, tb = tid >> 4;
    for (int ag = 0; ag < nA; ag += AG) {
      for (int bg = 0; bg < nB; bg += BG) {
        float acc[4][8];
#pragma unroll
        for (int q = 0; q < 4; q++)
#pragma unroll
          for (int jj = 0; jj < 8; jj++) acc[q][jj] = 0.f;
        for (int k0 = 0; k0 < d; k0 += KC) {
          for (int idx = tid; idx < AG * KC; idx += 256) {
            const int rr = idx / KC, kk = idx - rr * KC, aa = ag + rr;
            xa[rr][kk] = aa < nA ? a.x[(size_t)(base + 1 + 2 * aa) * d + k0 + kk] / nrm[2 * aa] : 0.f;
          }
          for (int idx = tid; idx < BG * KC; idx += 256) {
            const int rr = idx / KC, kk = idx - rr * KC, bb = bg + rr;
            xb[rr][kk] = bb < nB ? a.x[(size_t)(base + 2 + 2 * bb) * d + k0 + kk] / nrm[2 * bb + 1] : 0.f;
          }
          __syncthreads();
#pragma unroll
          for (int kk = 0; kk < KC; kk++) {
            float av[4], bv[8];
#pragma unroll
            for (int q = 0; q < 4; q++) av[q] = xa[ta * 4 + q][kk];
#pragma unroll
            for (int jj = 0; jj < 8; jj++) bv[jj] = xb[tb + 16 * jj][kk];
#pragma unroll
            for (int q = 0; q < 4; q++)
#pragma unroll
              for (int jj = 0; jj < 8; jj++) acc[q][jj] = fmaf(av[q], bv[jj], acc[q][jj]);
          }
          __syncthreads();
        }
#pragma unroll
        for (int q = 0; q < 4; q++) {
          float bvv = -INFINITY;
          int bi = 0x7fffffff;
#pragma unroll
          for (int jj = 0; jj < 8; jj++) {
            const int bb = bg + tb + 16 * jj;
            if (bb < nB && acc[q][jj] > bvv) {
              bvv = acc[q][jj];
              bi = bb;
            }
          }
          rbv[tb][ta * 4 + q] = bvv;
          rbi[tb][ta * 4 + q] = bi;
        }
        __syncthreads();
        if (tid < AG && ag + tid < nA) {
          const int aa = ag + tid;
          float v = bg == 0 ? -INFINITY : bestsim[aa];
          int vi = bg == 0 ? 0x7fffffff : best[aa];
          for (int t = 0; t < 16; t++) {
            const float cv = rbv[t][tid];
            const int ci = rbi[t][tid];
            if (cv > v || (cv == v && ci < vi)) {
              v = cv;
              vi = ci;
            }
          }
          bestsim[aa] = v;
          best[aa] = vi < nB ? vi : 0;  // only reachable with non-finite x
        }
        __syncthreads();
      }
    }
    // top-r of A by best similarity, ties to the lower A slot
    for (int aa = tid; aa < nA; aa += 256) {
      const float v = bestsim[aa];
      int rank = 0;
      for (int a2 = 0; a2 < nA; a2++) {
        const float v2 = bestsim[a2];
        rank += (v2 > v) || (v2 == v && a2 < aa);
      }
      chosen[aa] = rank < r;
    }
    __syncthreads();
    if (tid == 0) {
      int n = 0;
      for (int aa = 0; aa < nA; aa++)
        if (chosen[aa]) clist[n++] = aa;
    }
    __syncthreads();
    // size-weighted merge into each destination, sources in ascending order
    for (int idx = tid; idx < nB * d; idx += 256) {
      const int bb = idx / d, f = idx - bb * d;
      const size_t rowb = (size_t)(base + 2 + 2 * bb);
      float num = a.size[rowb] * a.x[rowb * d + f];
      float den = a.size[rowb];
      bool has = false;
      for (int q = 0; q < r; q++) {
        const int aa = clist[q];
        if (best[aa] == bb) {
          const size_t rowa = (size_t)(base + 1 + 2 * aa);
          num = num + a.size[rowa] * a.x[rowa * d + f];
          den = den + a.size[rowa];
          has = true;
        }
      }
      if (has) a.x[rowb * d + f] = num / den;
    }
    for (int bb = tid; bb < nB; bb += 256) {
      float den = a.size[base + 2 + 2 * bb];
      float s2 = a.isP ? sc[2 + 2 * bb] : 0.f;
      for (int q = 0; q < r; q++) {
        const int aa = clist[q];
        if (best[aa] == bb) {
          den = den + a.size[base + 1 + 2 * aa];
          if (a.isP) s2 = s2 + sc[1 + 2 * aa];
        }
      }
      tmpf[bb] = den;
      tmps[bb] = s2;
    }
    __syncthreads();
    for (int bb = tid; bb < nB; bb += 256) {
      a.size[base + 2 + 2 * bb] = tmpf[bb];
      if (a.isP) sc[2 + 2 * bb] = tmps[bb];
    }
    for (int q = tid; q < r; q += 256) {
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
    for (int k = tid; k < a.C; k += 256) lm = fmaxf(lm, lg[k]);
    lm = block_max256(lm, red);
    float s = 0.f;
    for (int k = tid; k < a.C; k += 256) s += expf(lg[k] - lm);
    s = block_sum256(s, red);
    const float c = 1.0f / s;
    fire = (a.delta < 1.0f) && (c >= a.delta);
    if (tid == 0 && a.tr_c) a.tr_c[tr_row] = c;
    if (fire) {
      for (int k = tid; k < a.C; k += 256) a.logits[(size_t)orig * a.C + k] = lg[k];
      if (tid == 0) a.exit_block[orig] = a.b;
    }
  }

  // ----------------------------------------------------------- prune --
  if (a.isP && !fire) {
    int ns = 0;
    for (int t = 1 + tid; t < T; t += 256) ns += keepf[t];
    ns = block_sum256_i(ns, ired);
    const int k = (int)floor(__dmul_rn(a.tau_eff, (double)ns));
    int keep_new[(AD_TMAX + 255) / 256];
#pragma unroll
    for (int u = 0; u < (AD_TMAX + 255) / 256; u++) {
      const int t = 1 + tid + u * 256;
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
    for (int u = 0; u < (AD_TMAX + 255) / 256; u++) {
      const int t = 1 + tid + u * 256;
      if (t < T) keepf[t] = keep_new[u];
    }
    __syncthreads();
  }

  int cnt = 0;
  for (int t = tid; t < T; t += 256) {
    const int kf = fire ? 0 : keepf[t];
    a.keep[base + t] = kf;
    cnt += kf;
  }
  cnt = block_sum256_i(cnt, ired);
  if (tid == 0) a.newlen[i] = cnt;
}

hipError_t launch_adapt(const AdaptArgs& a, hipStream_t s) {
  if (a.nlive_ub <= 0) return hipSuccess;
  if (a.n0 + 1 > AD_TMAX || a.d % KC != 0) return hipErrorInvalidValue;
  adapt_kernel<<<a.nlive_ub, 256, 0, s>>>(a);
  return hipGetLastError();
}

// --------------------------------------------------------- compaction --
__global__ __launch_bounds__(256) void compact_kernel(CompactArgs a) {
  const int i = blockIdx.x;
  const int nl = a.cnt->nlive;
  // Workgroup 0 always publishes the next counters, also when no sample is
  // live any more (the next block must see nlive = 0, not a stale value).
  if (i >= nl && i != 0) return;
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
  if (i == 0) {
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
  const int base = a.cu[i], T = a.cu[i + 1] - base;
  const int orig = a.live[i];
  if (tid == 0) {
    a.cu2[j] = off;
    a.live2[j] = orig;
  }
  const int nch = (T + 63) / 64;
  for (int c = wave; c < nch; c += 4) {
    const int t = c * 64 + lane;
    const unsigned long long msk = __ballot(t < T && a.keep[base + t]);
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
    const bool f = t < T && a.keep[base + t];
    const unsigned long long msk = __ballot(f);
    const int pos = __popcll(msk & ((1ull << lane) - 1ull));
    if (t < T) dsts[t] = f ? chunk_off[c] + pos : -1;
  }
  __syncthreads();
  const int d4 = a.d / 4;
  for (int idx = tid; idx < T * d4; idx += 256) {
    const int t = idx / d4, f = idx - t * d4;
    const int dj = dsts[t];
    if (dj >= 0)
      ((float4*)a.x2)[(size_t)(off + dj) * d4 + f] = ((const float4*)a.x)[(size_t)(base + t) * d4 + f];
  }
  for (int t = tid; t < T; t += 256) {
    const int dj = dsts[t];
    if (dj < 0) continue;
    a.size2[off + dj] = a.size[base + t];
    a.origin2[off + dj] = a.origin[base + t];
    if (a.tr_ids)
      a.tr_ids[((size_t)(a.b - 1) * a.B + orig) * (a.n0 + 1) + dj] = a.origin[base + t];
  }
}

hipError_t launch_compact(const CompactArgs& a, hipStream_t s) {
  if (a.nlive_ub <= 0) return hipSuccess;
  if (a.n0 + 1 > AD_TMAX || a.d % 4 != 0) return hipErrorInvalidValue;
  compact_kernel<<<a.nlive_ub, 256, 0, s>>>(a);
  return hipGetLastError();
}

}  // namespace fusion
