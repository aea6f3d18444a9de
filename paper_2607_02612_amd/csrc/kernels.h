// Host-side launchers of the gfx950 kernels (internal to the library).
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "common.h"

namespace fusion {

// Epilogue of the token GEMMs  C[M,N] = A[M,K] . W[N,K]^T.
enum EpiMode {
  EPI_STORE = 0,  // out(T)[r, n]  = acc + bias[n]
  EPI_GELU = 1,   // out(T)[r, n]  = GELU(acc + bias[n])
  EPI_RESID = 2,  // x(f32)[p, n] = x[p, n] + (acc + bias[n]), p = rows ? rows[r] : r
  EPI_F32 = 3,    // out(f32)[rows ? rows[r] : r, n] = acc + bias[n]
  EPI_PATCH = 4   // x(f32)[s (n0+1) + 1 + j, n] = (acc + bias[n]) + pos[1 + j, n],
                  //   r = s n0 + j
};

struct Epi {
  int mode;
  void* out;
  int ldo;
  const float* bias;
  const int* rows;  // EPI_F32 scatter map / EPI_RESID row map of x (optional)
  const float* pos; // EPI_PATCH
  int n0;           // EPI_PATCH
};

// Row count: *M_dev when non-null, else M_host.  M_ub bounds the grid.
template <typename T>
hipError_t launch_gemm(const T* A, int lda, const T* W, int N, int K,
                       const int* M_dev, int M_host, int M_ub, const Epi& e,
                       hipStream_t s);

template <typename T>
hipError_t launch_patchify(const float* img, T* out, int B, int C, int S,
                           int p, hipStream_t s);

// The fp32 residual stream x keeps every token in the physical row it was
// created in (merged tokens are updated in place); packed row r of the
// current state lives in physical row rmap[r].  Compaction repacks rmap,
// size and origin, not x.
//
// State at the start of a run: unit sizes, origin ids, identity row map,
// cu/live maps, CLS rows of x, zeroed token counts.
hipError_t launch_init(float* x, int* rmap, float* size, int* origin, int* cu, int* live,
                       LiveCounts* cnt, int* token_counts, const float* cls,
                       const float* pos, int B, int n0, int d, int L,
                       hipStream_t s);

// LayerNorm of packed rows, read through the row map (cls_only = 0: rows
// 0..M-1 -> out rows 0..M-1; cls_only = 1: row cu[i] of live sample i -> out
// row i).  When exit_block is
// non-null (final head), also writes exit_block[live[i]] = L.
template <typename T>
hipError_t launch_layernorm(const float* x, const int* rmap, const float* g, const float* b,
                            T* out, int d, const LiveCounts* cnt,
                            const int* cu, const int* live, int cls_only,
                            int rows_ub, int* exit_block, int L, hipStream_t s);

// LayerNorm of the size-weighted mean of each live sample's patch rows
// (pooled exit heads): out[i] = LN(sum_t s_t x_t / sum_t s_t).
template <typename T>
hipError_t launch_pool_ln(const float* x, const int* rmap, const float* size, const int* cu,
                          const LiveCounts* cnt, const float* g, const float* b,
                          T* out, int d, int nlive_ub, hipStream_t s);

struct AttnArgs {
  const void* qkv;  // T [M, 3d]
  const float* size;
  const int* cu;
  const int* live;
  const LiveCounts* cnt;
  int H, dh, d;
  float scale;
  int prop_attn;
  void* out;           // T [M, d]
  float* cls_scores;   // [nlive, H, tmax] or null
  int tmax;
  int* token_counts;   // [B, L]: written for head 0
  int L, b0;           // layers, 0-based block
  int nlive_ub, T_ub;
};
template <typename T>
hipError_t launch_attention(const AttnArgs& a, hipStream_t s);

struct AdaptArgs {
  float* x;
  const int* rmap;  // packed row -> physical row of x
  float* size;
  const int* origin;
  const int* cu;
  const int* live;
  const LiveCounts* cnt;
  int d, H, n0, C, L, B;
  int b;  // 1-based block
  int isM, isE, isP;
  int merge_rule;  // 0: budget, 1: fraction of the candidate pairs
  int prune_rule;  // 0: CLS-attention scores, 1: learned scorer
  const float* prune_w;  // [d] (learned scorer)
  const float* prune_b;  // [1]
  const float* router_w;
  const float* router_b;
  const int* r_fixed;  // optional [nlive]: merge counts given by the caller (no router)
  int r_b;
  double rho;
  const float* head_buf;  // [nlive, C] exit-head logits
  float delta;
  float* logits;
  int* exit_block;
  const float* cls_scores;
  int tmax;
  double tau_eff;
  int* keep;    // [M] row flags
  int* newlen;  // [nlive]
  int* tr_r;
  float* tr_m;
  float* tr_c;
  int* tr_merge;
  int nlive_ub;
  int T_ub;  // host bound on the tokens of every live sample (CLS included)
  // optional workspace [nlive_ub][AD_SIM_STRIDE]: best-match similarity and
  // index per A token, computed by a separate kernel for long samples
  float* sim_v;
  int* sim_i;
};
constexpr int AD_SIM_STRIDE = 320;  // A tokens of the longest size class (640 / 2)
hipError_t launch_adapt(const AdaptArgs& a, hipStream_t s);

struct CompactArgs {
  const float* x;
  const int* rmap;  // packed row -> physical row of x
  const float* size;
  const int* origin;
  const int* cu;
  const int* live;
  const LiveCounts* cnt;
  const int* keep;
  const int* newlen;
  int* rmap2;
  float* size2;
  int* origin2;
  int* cu2;
  int* live2;
  LiveCounts* cnt2;
  int d, n0, B, b;
  int* tr_ids;
  int nlive_ub;
  // optional: LayerNorm of every moved row with (ln_g, ln_b) into ln_out
  // (storage type T of the precision path), i.e. the next block's LN1
  const float* ln_g;
  const float* ln_b;
  void* ln_out;
};
template <typename T>
hipError_t launch_compact(const CompactArgs& a, hipStream_t s);

// Scratch of the kernel-level entry points: live map and row map set to the
// identity, live counts (nlive = B, M rows).
hipError_t launch_step_init(int* live, int B, int* rmap, int M, LiveCounts* cnt,
                            hipStream_t s);

// Error channel of the C ABI (message returned by fusion_last_error).
int api_fail(int code, const char* msg);

// Copy of the packed state for diagnostics.
hipError_t launch_copy_state(const float* x, const int* rmap, const int* cu, const int* live,
                             const LiveCounts* cnt, float* x_out, int* cu_out,
                             int* live_out, int d, int rows_ub, int nlive_ub,
                             hipStream_t s);

}  // namespace fusion
