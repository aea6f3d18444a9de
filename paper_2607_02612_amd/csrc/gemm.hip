// Token GEMMs C[M,N] = A[M,K] . W[N,K]^T with fused epilogues (bias, GELU,
// residual add into the fp32 stream, patch-embedding scatter, fp32 logits).
//
// bf16 path: MFMA v_mfma_f32_32x32x16_bf16 on 128x128 tiles staged through
// LDS, fp32 accumulation.  fp32 path: LDS-tiled VALU FMA (no rounding).
// Rows are the packed live tokens of all samples, so ragged lengths are
// invisible here: M is read from the device counters and the grid is sized
// for an upper bound (tiles past M return at once).
#include "kernels.h"

#include <type_traits>

namespace fusion {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

template <typename T>
__device__ __forceinline__ void epilogue(const Epi& e, int r, int n, float acc) {
  switch (e.mode) {
    case EPI_STORE:
      ((T*)e.out)[(size_t)r * e.ldo + n] = St<T>::put(acc + e.bias[n]);
      break;
    case EPI_GELU:
      ((T*)e.out)[(size_t)r * e.ldo + n] = St<T>::put(gelu_erf(acc + e.bias[n]));
      break;
    case EPI_RESID: {
      float* p = (float*)e.out + (size_t)(e.rows ? e.rows[r] : r) * e.ldo + n;
      *p = *p + (acc + e.bias[n]);
      break;
    }
    case EPI_F32: {
      const int orow = e.rows ? e.rows[r] : r;
      ((float*)e.out)[(size_t)orow * e.ldo + n] = acc + e.bias[n];
      break;
    }
    case EPI_PATCH: {
      const int s = r / e.n0, j = r - s * e.n0;
      const size_t xr = (size_t)s * (e.n0 + 1) + 1 + j;
      ((float*)e.out)[xr * e.ldo + n] =
          (acc + e.bias[n]) + e.pos[(size_t)(1 + j) * e.ldo + n];
      break;
    }
  }
}

// ------------------------------------------------------------ fp32 VALU --
template <typename T>
__global__ __launch_bounds__(256) void gemm_valu(const T* __restrict__ A,
                                                 int lda,
                                                 const T* __restrict__ W,
                                                 int N, int K,
                                                 const int* M_dev, int M_host,
                                                 Epi e) {
  const int M = M_dev ? *M_dev : M_host;
  const int m0 = blockIdx.x * 64, n0 = blockIdx.y * 64;
  if (m0 >= M) return;
  __shared__ float As[16][68];
  __shared__ float Ws[16][68];
  const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
  float acc[4][4];
#pragma unroll
  for (int i = 0; i < 4; i++)
#pragma unroll
    for (int j = 0; j < 4; j++) acc[i][j] = 0.f;
  for (int k0 = 0; k0 < K; k0 += 16) {
    for (int idx = threadIdx.x; idx < 64 * 16; idx += 256) {
      const int r = idx >> 4, kk = idx & 15;
      const int gk = k0 + kk;
      const int gr = m0 + r, gn = n0 + r;
      As[kk][r] = (gr < M && gk < K) ? St<T>::get(A[(size_t)gr * lda + gk]) : 0.f;
      Ws[kk][r] = (gn < N && gk < K) ? St<T>::get(W[(size_t)gn * K + gk]) : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < 16; kk++) {
      float a[4], w[4];
#pragma unroll
      for (int i = 0; i < 4; i++) {
        a[i] = As[kk][ty * 4 + i];
        w[i] = Ws[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++) acc[i][j] = fmaf(a[i], w[j], acc[i][j]);
    }
    __syncthreads();
  }
#pragma unroll
  for (int i = 0; i < 4; i++) {
    const int r = m0 + ty * 4 + i;
    if (r >= M) continue;
#pragma unroll
    for (int j = 0; j < 4; j++) {
      const int n = n0 + tx * 4 + j;
      if (n < N) epilogue<T>(e, r, n, acc[i][j]);
    }
  }
}

// ------------------------------------------------------------ bf16 MFMA --
// MBx128 output tile per workgroup (MB = 256: 8 waves in a 4x2 grid; 128: 4
// waves, 2x2; 64: 2 waves side by side), each wave a 64x64 sub-tile of 2x2
// v_mfma_f32_32x32x16_bf16 blocks; launches with few 64-row tiles split
// each into 4 waves of 32x64 (1x2 blocks) instead, which changes no result.
//
// K is consumed in steps of KSV = 32 through a ring of three LDS stages
// (64-wide steps with two stages measured slower on every shape, long K
// included).  A and W tiles reach LDS through the gfx950 asynchronous
// global->LDS path (global_load_lds_dwordx4): each wave-wide instruction
// writes 64 lanes x 16 bytes contiguously, i.e. 16 rows of 64 bytes,
// without passing through VGPRs, so later K steps are in
// flight while the matrix cores work on the current one (two or three
// workgroups share a CU and cover each other's load latency).  The loads
// are issued from inline assembly and their completion is awaited with
// explicit vmcnt counts (a compiler-visible LDS DMA would make every LDS
// read wait for all outstanding loads).  Each load names a wave-uniform
// operand base in SGPRs and a per-lane 32-bit byte offset, and the K loop is
// unrolled by the three ring stages, so that the loop's address arithmetic
// is scalar and the LDS reads take immediate offsets: no vector ALU work is
// left in the K loop (fc1 + GELU, which is bound by vector instruction
// issue, ran 11 % faster than with per-lane 64-bit pointers).  The 16-byte chunks of a staged row
// are XOR-permuted by (row / 4) % 4, which makes the per-lane 16-byte
// operand reads of 16 consecutive rows hit 16 disjoint bank groups.  Rows
// past M or N are clamped to the last valid row for the loads (every
// address stays in bounds) and masked in the epilogue.
//
// Epilogue: the accumulators start at the bias, and every load the epilogue
// needs (residual or position rows) is issued as one batch; for the staged
// fp32 epilogues the first round's row-map entries and addend rows are
// fetched during the last two K steps.  bf16 outputs are staged through LDS
// (the drained K ring) so that global stores are whole 256-byte row
// segments instead of 16-byte pieces of 32 different rows; the fp32
// residual update and the patch embedding are staged the same way as fp32
// rows (512-byte segments), on tiles of up to 128 rows; fp32 logits and
// 256-row tiles write directly.
//
// Tile order: blocks are dispatched round-robin over the 8 XCDs (block id %
// 8); the linear id is remapped so that each XCD walks whole row panels (all
// N tiles of one M tile back to back) and reuses the A panel in its own L2.
//
// Operand layout of v_mfma_f32_32x32x16_bf16 (64 lanes): lane l supplies
// A[row l%32][k 8*(l/32) .. +7] and B[k 8*(l/32) .. +7][col l%32]; result
// element q of lane l is C[8*(q/4) + 4*(l/32) + q%4][l%32].
constexpr int NB = 128;
constexpr int NXCD = 8;
constexpr long THIN_TILES = 768;

// 16-byte chunk c of staged row r (64-byte rows: four chunks)
__device__ __forceinline__ int kslot(int r, int c) { return c ^ ((r >> 2) & 3); }

// 16-byte store per lane: a wave-uniform 64-bit base in SGPRs plus the
// lane's 32-bit byte offset
typedef unsigned u32x4_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void st16s(const void* sbase, unsigned voff, u32x4_t v) {
  asm volatile("global_store_dwordx4 %0, %1, %2" :: "v"(voff), "v"(v), "s"(sbase) : "memory");
}
// global -> LDS copy of 16 bytes per lane: a wave-uniform 64-bit base in
// SGPRs plus the lane's 32-bit byte offset (advancing to the next K step is
// scalar arithmetic); the LDS destination is the wave-uniform m0
__device__ __forceinline__ void dma16s(const void* sbase, unsigned voff, unsigned lds_byte_addr) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(voff), "s"(sbase), "s"(__builtin_amdgcn_readfirstlane(lds_byte_addr))
               : "memory", "m0");
}
template <int N>
__device__ __forceinline__ void wait_vm() {
  asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory");
}

// MB = 256, 128 or 64 rows per tile; each wave owns WR * 32 rows x 64
// columns (WR = 2: 2 x 2 MFMA blocks, WR = 1: 1 x 2), the waves in a grid of
// MB / (32 WR) rows x 2 columns.  Every layout accumulates each output
// element over the same 16-wide K pieces in the same order from the same
// bias start, so the results do not depend on MB or WR.  KSV = K step (32).
template <int EPI, int MB, int KSV, int WR>
__global__ __launch_bounds__(MB / (32 * WR) * 128, MB == 128 ? 3 : 1) void gemm_mfma_bf16(
    const bf16_t* __restrict__ A, int lda, const bf16_t* __restrict__ W,
    int N, int K, const int* M_dev, int M_host, int n_mt, Epi e) {
  static_assert(KSV == 32, "K step of 32");
  constexpr int KS = KSV, NSTG = 3;
  constexpr int ROWB = KS * 2;                        // bytes per staged row
  constexpr int CPR = KS / 8;                         // 16-byte chunks per staged row
  constexpr int RPI = 64 / CPR;                       // rows per DMA instruction
  static_assert(WR == 1 || WR == 2, "32 or 64 rows per wave");
  constexpr int WMR = 32 * WR;                        // rows per wave
  constexpr int NWV = MB / WMR * 2;                   // waves
  constexpr int NT = NWV * 64;                        // threads
  constexpr int STGB = (MB + NB) * ROWB;              // bytes per stage
  constexpr int DMA_PER_WAVE = (MB + NB) / RPI / NWV; // DMA instructions per wave and stage
  static_assert((MB + NB) / RPI % NWV == 0, "stage split");
  const int M = M_dev ? *M_dev : M_host;
  const int n_nt = (N + NB - 1) / NB;
  const int id = blockIdx.x;
  const int xcd = id % NXCD, local = id / NXCD;
  const int mt = (local / n_nt) * NXCD + xcd, nt = local % n_nt;
  const int m0 = mt * MB, n0 = nt * NB;
  if (mt >= n_mt || m0 >= M) return;
  __shared__ __attribute__((aligned(16))) char smem[NSTG * STGB];
  const unsigned lds0 = (unsigned)(uintptr_t)(__attribute__((address_space(3))) void*)smem;
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6), lane = tid & 63;
  const int wm = wave >> 1, wn = wave & 1;
  // the accumulators start at the bias of their columns (lane l owns columns
  // n0 + wn 64 + 32 j + 8 (q / 4) + 4 (l / 32) + q % 4; columns past N, never
  // stored, take a clamped bias), so no epilogue adds it
  // (the column base is clamped as a whole: with N % 8 == 0 the lane
  // halves' columns c and c + 4 stay inside the bias vector; each
  // accumulator set loads its own copy, which costs no vector ALU moves)
  f32x16_t acc[WR][2];
  const float* bias_l = e.bias + 4 * (lane >> 5);
#pragma unroll
  for (int j = 0; j < 2; j++)
#pragma unroll
    for (int q4 = 0; q4 < 4; q4++) {
      const int cb = min(n0 + wn * 64 + j * 32 + 8 * q4, N - 8);
#pragma unroll
      for (int i = 0; i < WR; i++) {
        const float4 bv = *(const float4*)(bias_l + cb);
        acc[i][j][4 * q4 + 0] = bv.x;
        acc[i][j][4 * q4 + 1] = bv.y;
        acc[i][j][4 * q4 + 2] = bv.z;
        acc[i][j][4 * q4 + 3] = bv.w;
      }
    }

  // this lane's source row and LDS slot for each of the wave's DMA
  // instructions (8-row blocks: A rows first, then W rows)
  // per DMA instruction: a wave-uniform base (A or W) and LDS slot, and the
  // lane's byte offset from that base (rows past M or N clamped)
  const bf16_t* sbase[DMA_PER_WAVE];
  unsigned voff[DMA_PER_WAVE];
  unsigned dst[DMA_PER_WAVE];
#pragma unroll
  for (int u = 0; u < DMA_PER_WAVE; u++) {
    const int q = wave * DMA_PER_WAVE + u;
    const bool isA = q < MB / RPI;
    const int r = (isA ? q : q - MB / RPI) * RPI + lane / CPR;
    const int chunk = kslot(r, lane % CPR);
    if (isA) {
      const int gr = min(m0 + r, M - 1);
      sbase[u] = A;
      voff[u] = (unsigned)(((size_t)gr * lda + chunk * 8) * 2);
      dst[u] = q * RPI * ROWB;
    } else {
      const int gr = min(n0 + r, N - 1);
      sbase[u] = W;
      voff[u] = (unsigned)(((size_t)gr * K + chunk * 8) * 2);
      dst[u] = MB * ROWB + (q - MB / RPI) * RPI * ROWB;
    }
  }
  const int nk = K / KS;
#pragma unroll
  for (int st = 0; st < NSTG - 1; st++)
    if (st < nk) {
#pragma unroll
      for (int u = 0; u < DMA_PER_WAVE; u++)
        dma16s(sbase[u] + st * KS, voff[u], lds0 + st * STGB + dst[u]);
    }
  // staged residual / patch epilogue: the first round's row-map entries and
  // addend rows are fetched during the last two K steps, so that their
  // latency overlaps the final MFMAs
  constexpr bool STAGED = (EPI == EPI_RESID || EPI == EPI_PATCH) && MB <= 128;
  constexpr int RR = NSTG * STGB >= MB * NB * 4 ? MB : 64;  // rows per epilogue round
  constexpr int PER = RR * (NB / 4) / NT;                   // 16-byte pieces per thread
  float4 xpre[STAGED ? PER : 1];
  int ppre[STAGED ? PER : 1];
  auto row_map = [&](int rb, int* prow) {
    // one uniform branch for the whole batch: a select per entry would make
    // each load wait for every earlier memory access of the wave
    if (EPI == EPI_RESID && e.rows) {
#pragma unroll
      for (int k = 0; k < PER; k++)
        prow[k] = e.rows[min(m0 + rb + (tid + k * NT) / (NB / 4), M - 1)];
    } else {
#pragma unroll
      for (int k = 0; k < PER; k++) prow[k] = min(m0 + rb + (tid + k * NT) / (NB / 4), M - 1);
    }
  };
  auto addend = [&](int rb, const int* prow, float4* xv) {
    // the residual row (x += ...) or, for the patch embedding, the position
    // embedding of patch token 1 + j, whose output row is s (n0 + 1) + 1 + j
    // for packed row r = s n0 + j
#pragma unroll
    for (int k = 0; k < PER; k++) {
      const int idx = tid + k * NT;
      const int r = idx / (NB / 4), ch = idx % (NB / 4);
      const int m = min(m0 + rb + r, M - 1), n = min(n0 + ch * 4, N - 4);
      if (EPI == EPI_RESID) {
        xv[k] = *(const float4*)((const float*)e.out + (size_t)prow[k] * e.ldo + n);
      } else {
        const int pj = m - (m / e.n0) * e.n0;
        xv[k] = *(const float4*)(e.pos + (size_t)(1 + pj) * e.ldo + n);
      }
    }
  };
  // one K step; ST = kt % NSTG is a template argument so that the LDS
  // offsets of the stage are immediates
  auto kstep = [&](int kt, auto st_c) {
    constexpr int ST = decltype(st_c)::value;
    // stage kt has landed once at most the later stages are outstanding
    if (NSTG > 2 && kt + NSTG - 2 < nk)
      wait_vm<DMA_PER_WAVE * (NSTG - 2)>();
    else
      wait_vm<0>();
    __syncthreads();
    const int kn = kt + NSTG - 1;
    if (kn < nk) {
      constexpr int SN = (ST + NSTG - 1) % NSTG;
#pragma unroll
      for (int u = 0; u < DMA_PER_WAVE; u++)
        dma16s(sbase[u] + kn * KS, voff[u], lds0 + SN * STGB + dst[u]);
    }
    if constexpr (STAGED) {
      if (kt == max(nk - 2, 0)) row_map(0, ppre);
      if (kt == nk - 1) addend(0, ppre, xpre);
    }
    const char* Ab = smem + ST * STGB;
    const char* Bb = Ab + MB * ROWB;
#pragma unroll
    for (int ks = 0; ks < KS; ks += 16) {
      bf16x8_t a[2], b[2];
      const int c = (ks >> 3) + (lane >> 5);
#pragma unroll
      for (int i = 0; i < WR; i++) {
        const int r = wm * WMR + i * 32 + (lane & 31);
        a[i] = *(const bf16x8_t*)(Ab + r * ROWB + (kslot(r, c) << 4));
      }
#pragma unroll
      for (int j = 0; j < 2; j++) {
        const int r = wn * 64 + j * 32 + (lane & 31);
        b[j] = *(const bf16x8_t*)(Bb + r * ROWB + (kslot(r, c) << 4));
      }
      // transposed product: acc[i][j] holds C^T, so lane l owns output row
      // m = .. + (l % 32) and columns n = .. + 8 (q / 4) + 4 (l / 32) + q % 4
#pragma unroll
      for (int i = 0; i < WR; i++)
#pragma unroll
        for (int j = 0; j < 2; j++)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(b[j], a[i], acc[i][j], 0, 0, 0);
    }
  };
  static_assert(NSTG == 3, "the K loop is unrolled by three stages");
  for (int kt = 0; kt < nk; kt += NSTG) {
    kstep(kt, std::integral_constant<int, 0>{});
    if (kt + 1 < nk) kstep(kt + 1, std::integral_constant<int, 1>{});
    if (kt + 2 < nk) kstep(kt + 2, std::integral_constant<int, 2>{});
  }

  if (EPI == EPI_STORE || EPI == EPI_GELU) {
    // bf16 tile -> LDS -> global, 16 lanes per 256-byte row segment.  After
    // GELU (bound by vector instruction issue) the staged rows are 256
    // bytes padded to 272, so that every staging address is one per-lane
    // base plus an immediate; the plain store keeps unpadded rows with the
    // 16-byte chunk c of row r at c ^ (r % 16) (conflict-free, and faster
    // for the 256-row QKV tiles)
    constexpr bool PAD = EPI == EPI_GELU;
    constexpr int SROW = PAD ? NB * 2 + 16 : NB * 2;
    static_assert(MB * SROW <= NSTG * STGB, "epilogue staging fits");
    __syncthreads();
    char* sl = smem + (wm * WMR + (lane & 31)) * SROW + (PAD ? wn * 128 + (lane >> 5) * 8 : 0);
#pragma unroll
    for (int j = 0; j < 2; j++) {
#pragma unroll
      for (int q4 = 0; q4 < 4; q4++) {
        // (N % 8 == 0: the lane halves' columns c and c + 4 are on the
        // same side of N, so the check is uniform)
        if (n0 + wn * 64 + j * 32 + 8 * q4 >= N) continue;
#pragma unroll
        for (int i = 0; i < WR; i++) {
          float v0 = acc[i][j][4 * q4 + 0], v1 = acc[i][j][4 * q4 + 1];
          float v2 = acc[i][j][4 * q4 + 2], v3 = acc[i][j][4 * q4 + 3];
          if (EPI == EPI_GELU) {
            v0 = gelu_erf(v0); v1 = gelu_erf(v1); v2 = gelu_erf(v2); v3 = gelu_erf(v3);
          }
          const uint2 pk = make_uint2(pack_bf16x2(v0, v1), pack_bf16x2(v2, v3));
          if (PAD) {
            *(uint2*)(sl + i * 32 * SROW + j * 64 + q4 * 16) = pk;
          } else {
            const int r = wm * WMR + i * 32 + (lane & 31);
            const int c = wn * 64 + j * 32 + 8 * q4 + 4 * (lane >> 5);
            *(uint2*)(smem + r * SROW + (((c >> 3) ^ (r & 15)) << 4) + ((c >> 2) & 1) * 8) = pk;
          }
        }
      }
    }
    __syncthreads();
    // lane: row tid / 16 + 16 it, 16-byte piece tid % 16; the stores take a
    // uniform row-block base in SGPRs plus the lane's 32-bit byte offset
    const unsigned lo = (unsigned)(((tid >> 4) * e.ldo + (tid & 15) * 8) * 2);
    const int mr = M - m0 - (tid >> 4);   // rows from the lane's first row to M
    const bool col_ok = n0 + (tid & 15) * 8 < N;
#pragma unroll
    for (int it = 0; it < MB * (NB / 8) / NT; it++) {
      const int r = (tid >> 4) + it * (NT / 16), cc = tid & 15;
      const u32x4_t v = PAD ? *(const u32x4_t*)(smem + r * SROW + cc * 16)
                            : *(const u32x4_t*)(smem + r * SROW + ((cc ^ (r & 15)) << 4));
      if (it * (NT / 16) < mr && col_ok)
        st16s((const bf16_t*)e.out + (size_t)(m0 + it * (NT / 16)) * e.ldo + n0, lo, v);
    }
    return;
  }
  if ((EPI == EPI_RESID || EPI == EPI_PATCH) && MB <= 128) {
    // residual update (and patch embedding) through LDS: the accumulator
    // rows (bias included) are staged in fp32
    // (512-byte rows, 16-byte chunk c of row r at c ^ (r % 32)), then the
    // workgroup adds them to x with whole-row accesses (32 lanes per
    // 512-byte row segment) instead of 16-byte pieces of 32 rows per
    // instruction.  RR rows per round: the whole tile when the drained ring
    // holds it (64-row tiles), else rounds of 64 rows.
    float* x = (float*)e.out;
#pragma unroll
    for (int rb = 0; rb < MB; rb += RR) {
      __syncthreads();
      if (wm * WMR >= rb && wm * WMR < rb + RR) {
#pragma unroll
        for (int j = 0; j < 2; j++) {
#pragma unroll
          for (int i = 0; i < WR; i++) {
            const int r = wm * WMR + i * 32 + (lane & 31) - rb;
#pragma unroll
            for (int q4 = 0; q4 < 4; q4++) {
              const int c = wn * 64 + j * 32 + 8 * q4 + 4 * (lane >> 5);
              *(float4*)(smem + r * (NB * 4) + (((c >> 2) ^ (r & 31)) << 4)) =
                  make_float4(acc[i][j][4 * q4 + 0], acc[i][j][4 * q4 + 1],
                              acc[i][j][4 * q4 + 2], acc[i][j][4 * q4 + 3]);
            }
          }
        }
      }
      __syncthreads();
      float4 xv[PER];
      int prow[PER];
      if (rb == 0) {
#pragma unroll
        for (int k = 0; k < PER; k++) {
          xv[k] = xpre[k];
          prow[k] = ppre[k];
        }
      } else {
        row_map(rb, prow);
        addend(rb, prow, xv);
      }
#pragma unroll
      for (int k = 0; k < PER; k++) {
        const int idx = tid + k * NT;
        const int r = idx / (NB / 4), ch = idx % (NB / 4);
        const int m = m0 + rb + r, n = n0 + ch * 4;
        const float4 sv = *(const float4*)(smem + r * (NB * 4) + ((ch ^ (r & 31)) << 4));
        if (m < M && n < N) {
          size_t orow = (size_t)prow[k];
          if (EPI == EPI_PATCH) {
            const int sidx = m / e.n0;
            orow = (size_t)sidx * (e.n0 + 1) + 1 + (m - sidx * e.n0);
          }
          *(float4*)(x + orow * e.ldo + n) =
              make_float4(sv.x + xv[k].x, sv.y + xv[k].y, sv.z + xv[k].z, sv.w + xv[k].w);
        }
      }
    }
    return;
  }
  // residual update (other tile heights), fp32 logits (row scatter) and the
  // patch embedding: direct vector accesses
#pragma unroll
  for (int i = 0; i < WR; i++) {
    const int m = m0 + wm * WMR + i * 32 + (lane & 31);
    if (m >= M) continue;
    size_t orow = (size_t)m;
    int pj = 0;
    if (EPI == EPI_F32 || EPI == EPI_RESID) orow = e.rows ? (size_t)e.rows[m] : (size_t)m;
    if (EPI == EPI_PATCH) {
      const int sidx = m / e.n0;
      pj = m - sidx * e.n0;
      orow = (size_t)sidx * (e.n0 + 1) + 1 + pj;
    }
#pragma unroll
    for (int j = 0; j < 2; j++) {
      // all loads of the column block first (the residual or position
      // rows), then the arithmetic and the stores
      float4 xv[4];
#pragma unroll
      for (int q4 = 0; q4 < 4; q4++) {
        const int nb = min(n0 + wn * 64 + j * 32 + 8 * q4 + 4 * (lane >> 5), N - 4);
        if (EPI == EPI_RESID) xv[q4] = *(const float4*)((const float*)e.out + orow * e.ldo + nb);
        if (EPI == EPI_PATCH) xv[q4] = *(const float4*)(e.pos + (size_t)(1 + pj) * e.ldo + nb);
      }
#pragma unroll
      for (int q4 = 0; q4 < 4; q4++) {
        const int nb = n0 + wn * 64 + j * 32 + 8 * q4 + 4 * (lane >> 5);
        if (nb >= N) continue;
        const float v0 = acc[i][j][4 * q4 + 0], v1 = acc[i][j][4 * q4 + 1];
        const float v2 = acc[i][j][4 * q4 + 2], v3 = acc[i][j][4 * q4 + 3];
        float4* po = (float4*)((float*)e.out + orow * e.ldo + nb);
        if (EPI == EPI_RESID) {
          *po = make_float4(xv[q4].x + v0, xv[q4].y + v1, xv[q4].z + v2, xv[q4].w + v3);
        } else if (EPI == EPI_F32) {
          *po = make_float4(v0, v1, v2, v3);
        } else {  // EPI_PATCH: + position embedding of token 1 + pj
          *po = make_float4(v0 + xv[q4].x, v1 + xv[q4].y, v2 + xv[q4].z, v3 + xv[q4].w);
        }
      }
    }
  }
}


template <>
hipError_t launch_gemm<float>(const float* A, int lda, const float* W, int N,
                              int K, const int* M_dev, int M_host, int M_ub,
                              const Epi& e, hipStream_t s) {
  if (M_ub <= 0) return hipSuccess;
  dim3 grid((M_ub + 63) / 64, (N + 63) / 64);
  gemm_valu<float><<<grid, 256, 0, s>>>(A, lda, W, N, K, M_dev, M_host, e);
  return hipGetLastError();
}

template <>
hipError_t launch_gemm<bf16_t>(const bf16_t* A, int lda, const bf16_t* W,
                               int N, int K, const int* M_dev, int M_host,
                               int M_ub, const Epi& e, hipStream_t s) {
  if (M_ub <= 0) return hipSuccess;
  // The K steps need K % 32 == 0 and 16-byte aligned rows; the vector
  // epilogues need N and the output stride to be multiples of 8 (bf16
  // outputs) or 4 (fp32 outputs).  The model creation rejects bf16 shapes
  // that do not satisfy this.
  if (K % 32 != 0 || lda % 8 != 0 || K <= 0) return hipErrorInvalidValue;
  if (N % 4 != 0 || e.ldo % 4 != 0) return hipErrorInvalidValue;
  // the loads take 32-bit byte offsets from the operand bases
  if ((size_t)M_ub * lda * 2 > 0xFFFFFFFFull || (size_t)N * K * 2 > 0xFFFFFFFFull)
    return hipErrorInvalidValue;
  if ((e.mode == EPI_STORE || e.mode == EPI_GELU) && (N % 8 != 0 || e.ldo % 8 != 0))
    return hipErrorInvalidValue;
  const int n_nt = (N + NB - 1) / NB;
  // tile rows: 256 (8 waves) when there are enough tiles to fill the CUs
  // several times over, 64 when 128-row tiles would leave CUs idle
  const bool small = (long)((M_ub + 127) / 128) * n_nt < 512;
  // K steps of 32 with three stages everywhere: 64-wide steps (two stages,
  // half the barriers) measured slower on every shape here, long K included
  // (not for the GELU epilogue, whose vector work overlaps better with
  // three 4-wave workgroups per CU than with two 8-wave ones)
  const bool big = e.mode != EPI_GELU &&
                   (long)((M_ub + 255) / 256) * n_nt >= 1024;
  const int mb = small ? 64 : big ? 256 : 128;
  const int n_mt = (M_ub + mb - 1) / mb;
  const int grid = (n_mt + NXCD - 1) / NXCD * NXCD * n_nt;
  // 32-row waves (twice the waves per tile) for 64-row tiles when the
  // launch has fewer tiles than the CUs hold at once
  const bool thin = small && (long)n_mt * n_nt < THIN_TILES;
#define FUSION_GEMM_LAUNCH(E)                                                                    \
  if (small && thin)                                                                            \
    gemm_mfma_bf16<E, 64, 32, 1><<<grid, 256, 0, s>>>(A, lda, W, N, K, M_dev, M_host, n_mt, e); \
  else if (small)                                                                               \
    gemm_mfma_bf16<E, 64, 32, 2><<<grid, 128, 0, s>>>(A, lda, W, N, K, M_dev, M_host, n_mt, e); \
  else if (big)                                                                                 \
    gemm_mfma_bf16<E, 256, 32, 2><<<grid, 512, 0, s>>>(A, lda, W, N, K, M_dev, M_host, n_mt, e); \
  else                                                                                          \
    gemm_mfma_bf16<E, 128, 32, 2><<<grid, 256, 0, s>>>(A, lda, W, N, K, M_dev, M_host, n_mt, e)
  switch (e.mode) {
    case EPI_STORE: FUSION_GEMM_LAUNCH(EPI_STORE); break;
    case EPI_GELU: FUSION_GEMM_LAUNCH(EPI_GELU); break;
    case EPI_RESID: FUSION_GEMM_LAUNCH(EPI_RESID); break;
    case EPI_F32: FUSION_GEMM_LAUNCH(EPI_F32); break;
    case EPI_PATCH: FUSION_GEMM_LAUNCH(EPI_PATCH); break;
    default: return hipErrorInvalidValue;
  }
#undef FUSION_GEMM_LAUNCH
  return hipGetLastError();
}

}  // namespace fusion
