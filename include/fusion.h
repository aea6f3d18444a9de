/*
 * fusion.h -- C ABI of the MI355X (gfx950) library for Fusion's staged
 * adaptive Vision Transformer inference: each block runs MHSA and MLP, then
 * token merging, then an exit check on the CLS token, then token pruning on
 * the samples that continue (Algorithm 1, Sec. III-B of the Fusion paper).
 *
 * Conventions for every entry point
 *   - Return value: FUSION_OK (0) or a negative fusion_status.  On error a
 *     thread-local message is available from fusion_last_error().
 *   - Arguments are validated on the host before anything is enqueued; an
 *     invalid call leaves device memory and the stream untouched.
 *   - "device" pointers are HIP device allocations (for example the
 *     data_ptr() of a torch tensor on the GPU); "host" pointers are ordinary
 *     CPU memory.  The library never frees memory it did not allocate.
 *   - fusion_run / fusion_run_traced are asynchronous on the given stream
 *     (a hipStream_t, or NULL for the default stream); outputs are valid once
 *     that stream is synchronised.  One model handle must not run on two
 *     streams at the same time (it owns one workspace).
 */
#ifndef FUSION_H
#define FUSION_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define FUSION_API __attribute__((visibility("default")))
#define FUSION_MAX_LAYERS 32

typedef struct fusion_model fusion_model; /* opaque */

typedef enum fusion_status {
  FUSION_OK = 0,
  FUSION_E_INVALID_ARG = -1, /* null pointer, out-of-range value */
  FUSION_E_BLOB = -2,        /* malformed or inconsistent weight blob */
  FUSION_E_CAPACITY = -3,    /* batch larger than the model's max_batch */
  FUSION_E_OOM = -4,         /* device allocation failed */
  FUSION_E_HIP = -5,         /* a HIP runtime call or launch failed */
  FUSION_E_STATE = -6        /* call not valid in the model's state */
} fusion_status;

/* Merge-count rules (Sec. III-C, Eq. 4-5), with m the router output and
 * rho the router strength (fusion_set_router_strength):
 *   BUDGET:   r = clamp(floor(2 rho m r_b + 1/2), 0, floor(N/2));
 *   FRACTION: r = min(floor(((rho m) N) / 2), floor(N/2)), the merge ratio
 *             m~ = rho m applied to the N/2 candidate pairs. */
enum { FUSION_MERGE_BUDGET = 0, FUSION_MERGE_FRACTION = 1 };
/* Token scores of the prune step (Eq. 8):
 *   CLS_ATTN: head-mean CLS-attention probability of the block (added up
 *             over merged tokens);
 *   LEARNED:  s_i = w . z_i + beta, a linear scorer on the hidden states
 *             after the block's merge (tensors prune_w [d], prune_b [1]). */
enum { FUSION_PRUNE_CLS_ATTN = 0, FUSION_PRUNE_LEARNED = 1 };
/* Exit-head kinds (Eq. 6 head_b; Sec. IV describes MLP heads):
 *   LINEAR:   LN + linear on the CLS token;
 *   CLS_MLP:  LN, linear to exit_hidden, exact GELU, linear to C, on CLS;
 *   POOL_MLP: the same MLP on sum_t s_t z_t / sum_t s_t over the patch
 *             tokens (token sizes s_t, CLS excluded; zero vector when no
 *             patch token is left). */
enum { FUSION_EXIT_LINEAR = 0, FUSION_EXIT_CLS_MLP = 1, FUSION_EXIT_POOL_MLP = 2 };

/* Static description of a model (filled by fusion_model_info or
 * fusion_blob_inspect). */
typedef struct fusion_info {
  int32_t img, patch, in_ch;   /* square image side, patch side, channels */
  int32_t d, heads, layers;    /* embedding width, heads, blocks L */
  int32_t mlp, classes;        /* MLP hidden width, classes C */
  int32_t n0;                  /* patch tokens N0 = (img/patch)^2 */
  int32_t precision;           /* 0 = fp32 path, 1 = bf16 path */
  int32_t prop_attn;           /* 1: attention scores += ln(token size) */
  int32_t max_batch;           /* 0 from fusion_blob_inspect */
  uint32_t merge_mask, exit_mask, prune_mask; /* bit b-1 <=> block b */
  int32_t n_exit;              /* number of exit heads |E| */
  int32_t exit_blocks[FUSION_MAX_LAYERS]; /* ascending, 1-based */
  int32_t r_b[FUSION_MAX_LAYERS];         /* merge budget per block */
  double tau_b[FUSION_MAX_LAYERS];        /* keep ratio per block */
  float delta[FUSION_MAX_LAYERS];         /* current threshold per exit head */
  double rho;                             /* current router strength */
  int32_t merge_rule;                     /* FUSION_MERGE_* */
  int32_t prune_rule;                     /* FUSION_PRUNE_* */
  int32_t exit_kind[FUSION_MAX_LAYERS];   /* FUSION_EXIT_* per block (exit blocks) */
  int32_t exit_hidden;                    /* hidden width of MLP exit heads, 0 if none */
} fusion_info;

/* Per-block decision record written by fusion_run_traced.  Every pointer is
 * a device buffer owned by the caller, indexed by the sample's position in
 * the input batch; entries the run does not reach are left untouched, so
 * the caller pre-fills them (e.g. with -1).  Any pointer may be NULL.
 *   r         int32 [L][B]          merge count of the block (merge blocks)
 *   m         float [L][B]          merge-router output m (merge blocks)
 *   c         float [L][B]          exit confidence max softmax (exit blocks)
 *   merge_dst int32 [L][B][N0+1]    at index = origin id of a token merged
 *                                   away in block b: origin id of the token
 *                                   it merged into
 *   ids       int32 [L][B][N0+1]    origin ids of the tokens that leave
 *                                   block b (after merge and prune), in
 *                                   sequence order; nothing for samples that
 *                                   exit at b
 * A token's origin id is its index in the initial N0+1 sequence (CLS = 0);
 * a merged token keeps the id of the token it merged into. */
typedef struct fusion_trace {
  int32_t* r;
  float* m;
  float* c;
  int32_t* merge_dst;
  int32_t* ids;
} fusion_trace;

/* Parse and check a weight blob on the host without touching the device.
 * blob: host, blob_bytes long (layout documented in the package's blob
 * writer: header, tensor table, fp32 data).  Fills *out (max_batch = 0).
 * Errors: FUSION_E_INVALID_ARG (null), FUSION_E_BLOB (bad magic, version,
 * sizes, tensor names/shapes/offsets). */
FUSION_API int fusion_blob_inspect(const void* blob, size_t blob_bytes,
                                   fusion_info* out);

/* Create a model on the current HIP device from a weight blob (the paper's
 * backbone plus merge routers, exit heads and final head; Sec. III-A).
 * blob: host memory, copied and converted (fp32 -> bf16 for matrix weights
 * on the bf16 path) during the call; the caller may free it afterwards.
 * max_batch: largest batch fusion_run will accept (1 .. 65536); the
 * workspace is sized for it, and max_batch * (N0 + 1) * d must stay below
 * 2^31 (the residual stream's element count) and max_batch * (N0 + 1) *
 * max(3 d, mlp, 3 p^2) operand bytes below 2^32 (the GEMMs address their
 * operands with 32-bit offsets; about 7,000 DeiT-S images at 224 x 224).
 * *out receives the handle.
 * Errors: FUSION_E_INVALID_ARG, FUSION_E_BLOB (before any device call),
 * FUSION_E_CAPACITY (max_batch beyond either limit),
 * FUSION_E_OOM, FUSION_E_HIP. */
FUSION_API int fusion_model_create(const void* blob, size_t blob_bytes,
                                   int max_batch, fusion_model** out);

/* Free every device allocation of the model (synchronises the device). */
FUSION_API int fusion_model_destroy(fusion_model* m);

/* Describe the model (host struct). */
FUSION_API int fusion_model_info(const fusion_model* m, fusion_info* out);

/* Exit thresholds delta_b of the exit rule c_b >= delta_b (Eq. 7), one per
 * exit head in ascending block order.  delta: host, n_exit values in
 * [0, 1]; a value >= 1 disables that head.  Applies to runs enqueued
 * afterwards.  Errors: FUSION_E_INVALID_ARG (null, count != |E|, NaN or out
 * of range). */
FUSION_API int fusion_set_exit_thresholds(fusion_model* m, const float* delta,
                                          int n_exit);

/* Router strength rho: the profile ratio of Eq. 5.  Merge blocks merge
 * r pairs by the model's merge rule (FUSION_MERGE_*); prune blocks
 * keep floor(tau' N) patch tokens with tau' = min(1, max(0, 1 - rho (1 -
 * tau_b))).  rho = 1 is the reference profile, rho = 0 disables merging and
 * pruning.  Range [0, 16].  A double, because the count expressions are
 * evaluated in IEEE double: a float would round a ratio such as 5/3 before
 * it enters them.  Errors: FUSION_E_INVALID_ARG. */
FUSION_API int fusion_set_router_strength(fusion_model* m, double rho);

/* Run Algorithm 1 on a batch.
 * images:       device, fp32 [batch][in_ch][img][img] (NCHW), read only.
 * batch:        1 .. max_batch.
 * logits:       device, fp32 [batch][classes]: the exit head's logits for
 *               samples that exit early, else the final head's.
 * exit_block:   device, int32 [batch]: 1-based block whose head produced the
 *               logits (layers if the sample ran every block).
 * token_counts: device, int32 [batch][layers]: tokens (CLS included)
 *               entering each block, 0 for blocks the sample skipped.
 * stream:       hipStream_t or NULL.
 * Errors: FUSION_E_INVALID_ARG, FUSION_E_CAPACITY, FUSION_E_HIP. */
FUSION_API int fusion_run(fusion_model* m, const float* images, int batch,
                          float* logits, int32_t* exit_block,
                          int32_t* token_counts, void* stream);

/* fusion_run plus the per-block decision record (trace: host struct of
 * device pointers, see fusion_trace). */
FUSION_API int fusion_run_traced(fusion_model* m, const float* images,
                                 int batch, float* logits,
                                 int32_t* exit_block, int32_t* token_counts,
                                 const fusion_trace* trace, void* stream);

/* Diagnostic: run the pipeline up to block `block` (1-based) and stop after
 * stage `stage` of that block (0: patch embedding, block ignored; 1: after
 * the attention residual; 2: after the MLP residual, before any merge, exit
 * or prune of that block).  Copies the packed fp32 hidden states of the
 * live samples to x_out (device, >= batch*(n0+1)*d floats; rows of live
 * sample j start at cu_out[j]) and cu_out (device int32, >= batch+1), and
 * the live sample ids to live_out (device int32, >= batch).  The host
 * receives the live count in *n_live (this call synchronises the stream).
 */
FUSION_API int fusion_debug_state(fusion_model* m, const float* images,
                                  int batch, int block, int stage,
                                  float* x_out, int32_t* cu_out,
                                  int32_t* live_out, int* n_live,
                                  void* stream);

/* Diagnostic (race proxy): fill the model's floating-point workspace (the
 * fp32 residual stream and token sizes, the activation, q|k|v, MLP, head and
 * CLS-score buffers) with NaN bytes, asynchronously on the stream.  A run
 * enqueued afterwards must give bit-identical outputs to an unpoisoned run:
 * every value a run reads is written earlier in the same run.  The integer
 * maps (row map, offsets, live map, counts, keep flags) are not touched.
 * Errors: FUSION_E_INVALID_ARG, FUSION_E_HIP. */
FUSION_API int fusion_debug_poison_workspace(fusion_model* m, void* stream);

/* Per-kernel timing for measurement: when enabled, runs record a pair of
 * HIP events around every launch on the run's stream and accumulate the
 * elapsed time per kernel kind once fusion_profile_read synchronises.
 * Enabling resets the totals. */
FUSION_API int fusion_profile_enable(fusion_model* m, int on);

/* Number of kernel kinds and the name of kind k (static string). */
FUSION_API int fusion_profile_kinds(void);
FUSION_API const char* fusion_profile_kind_name(int k);

/* Totals since enabling for kind k: milliseconds and launch count (host
 * outputs).  Synchronises the pending events. */
FUSION_API int fusion_profile_read(fusion_model* m, int k, double* total_ms,
                                   int64_t* launches);

/* ------------------------------------------------------------------------
 * Kernel-level entry points.  Each runs the kernels fusion_run launches for
 * one step of Algorithm 1 on caller-supplied buffers instead of a model's
 * workspace, so that the step can be checked (the GPU tests drive every
 * kernel this way, at random ragged lengths) or used on its own.
 *
 * Packed ragged layout: the rows of sample i are rows cu[i] .. cu[i+1]-1 of
 * every per-row buffer, CLS first; cu is a HOST array of batch + 1 offsets
 * with cu[0] = 0 and 1 .. 640 rows per sample (M = cu[batch] rows in all);
 * batch is 1 .. 65536.  Arguments are checked on the host before anything is
 * enqueued (FUSION_E_INVALID_ARG, nothing launched).  Calls with scratch
 * (all but fusion_test_gemm) allocate it for the call and synchronise the
 * stream before returning; fusion_test_gemm is asynchronous.
 * ------------------------------------------------------------------------ */

/* Ragged token state of a batch (all device pointers but cu). */
typedef struct fusion_ragged {
  float* x;               /* device fp32 [M][d] hidden states (row-major) */
  const float* size;      /* device fp32 [M] token sizes (read only) */
  const int32_t* origin;  /* device int32 [M] token ids (read only) */
  const int32_t* cu;      /* HOST int32 [batch + 1] row offsets */
  int32_t batch;
  int32_t d;              /* width: a multiple of 32, at most 768 */
} fusion_ragged;

/* Re-packed state after a step (Sec. III-C: N_b shrinks per sample), all
 * device buffers owned by the caller:
 *   rows   int32 [M]          input row of each output row (the fp32 rows
 *                             themselves are not moved)
 *   size   fp32  [M]          size of each output row's token
 *   origin int32 [M]          its id
 *   cu     int32 [batch + 1]  offsets of the surviving samples (first
 *                             n_live + 1 entries written)
 *   live   int32 [batch]      input index of each surviving sample
 *   counts int32 [2]          n_live, total output rows */
typedef struct fusion_packed_out {
  int32_t* rows;
  float* size;
  int32_t* origin;
  int32_t* cu;
  int32_t* live;
  int32_t* counts;
} fusion_packed_out;

/* Epilogues of fusion_test_gemm. */
enum { FUSION_EPI_STORE = 0, FUSION_EPI_GELU = 1, FUSION_EPI_RESID = 2, FUSION_EPI_F32 = 3 };

/* A token GEMM, the linear maps of Eq. 2 and the heads of Eq. 3 and Eq. 6:
 * acc[r][n] = sum_k A[r][k] W[n][k] + bias[n] (fp32 accumulation), then
 *   STORE: out[r][n] = acc (storage type: bf16 rounded to nearest even, or
 *          fp32);  GELU: out[r][n] = GELU(acc), exact-erf form (storage type);
 *   RESID: out[p][n] += acc, p = rows ? rows[r] : r (fp32 out);
 *   F32:   out[p][n]  = acc (fp32 out).
 * precision 1: A, W bf16 bit patterns (uint16), K % 32 == 0, lda % 8 == 0,
 * N and ldo multiples of 8 (STORE, GELU) or 4 (RESID, F32); precision 0:
 * fp32 operands.  A: device [M][lda]; W: device [N][K]; bias: device fp32
 * [N]; out: device [*][ldo]; rows: device int32 [M] or NULL.  Asynchronous.
 */
FUSION_API int fusion_test_gemm(int precision, const void* A, int lda, const void* W, int N,
                                int K, int M, const float* bias, int epi, void* out,
                                int ldo, const int32_t* rows, void* stream);

/* Multi-head self-attention of every sample over its own rows (Eq. 2), with
 * proportional attention when prop_attn = 1 (scores += ln(size of the key
 * token), the companion of size-weighted merging, Sec. III-C), and the
 * per-head CLS-attention rows that score tokens for pruning (Eq. 8).
 * qkv: device [M][3d] in the storage type (columns q | k | v, head-major);
 * size: device fp32 [M]; out: device [M][d] storage type; cls_scores:
 * device fp32 [batch][heads][tmax] (row h of sample i: softmax
 * probabilities of its CLS query, entries past the sample's rows untouched)
 * or NULL.  precision 1 needs 64-wide heads.  Synchronises the stream. */
FUSION_API int fusion_test_attention(int precision, const void* qkv, const float* size,
                                     const int32_t* cu, int batch, int heads, int d,
                                     int prop_attn, void* out, float* cls_scores, int tmax,
                                     void* stream);

/* Bipartite soft matching with size-weighted merging (Sec. III-C) of r[i]
 * token pairs in every sample, then re-compaction: the patch tokens
 * (rows 1..N) split into A = even and B = odd slots, cosine similarity of
 * the fp32 rows, best B per A (ties to the lowest B), the r A tokens with
 * the highest best similarity (ties to the lowest A) merge into their B:
 * dst = (s_dst x_dst + sum_a s_a x_a) / (s_dst + sum_a s_a), sizes add.
 * r: HOST int32 [batch], 0 <= r[i] <= floor(N_i / 2).  in->x is updated in
 * place (each destination row receives its merged value); the survivors,
 * in order, are described by *out.  merge_dst: device int32
 * [batch][id_stride] or NULL; entry [i][id of a merged-away token] receives
 * the id of the token it merged into (origin ids must lie in
 * 0 .. id_stride-1; others are not recorded).  Synchronises the stream. */
FUSION_API int fusion_test_merge(const fusion_ragged* in, const int32_t* r, int id_stride,
                                 int32_t* merge_dst, const fusion_packed_out* out,
                                 void* stream);

/* fusion_test_merge without any device allocation, for callers that cannot
 * allocate (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc).  Same arguments, checks and results as
 * fusion_test_merge.  Its scratch is a static device array of the library
 * (FUSION_NOALLOC_SCRATCH_BYTES, one per GPU, held until the process ends);
 * a call needs 12 bytes per row plus 16 per sample (each part rounded up to
 * 256 bytes), so batch 256 at 197 tokens takes about 0.6 MiB.  The call
 * makes no allocation and does not synchronise: it is asynchronous on the
 * stream like fusion_run (the host offsets and counts are copied in before
 * it returns).  Every call on one GPU shares that GPU's array: calls that
 * overlap (other streams, other threads) race, so serialise them.  Errors:
 * FUSION_E_CAPACITY when the call needs more scratch than the array holds,
 * otherwise as fusion_test_merge. */
#define FUSION_NOALLOC_SCRATCH_BYTES (1u << 20)
FUSION_API int fusion_test_merge_noalloc(const fusion_ragged* in, const int32_t* r,
                                         int id_stride, int32_t* merge_dst,
                                         const fusion_packed_out* out, void* stream);

/* Exit check (Eq. 7; optional), top-k pruning of the samples that continue
 * (Eq. 8) and re-compaction.  Token scores: the head mean of CLS-attention
 * probabilities, scores = device fp32 [batch][heads][tmax] laid out as
 * fusion_test_attention writes them; or, when scores is NULL, the learned
 * linear scorer w . x_t + beta (prune_w: device fp32 [d], prune_b: [1]).
 * Each continuing sample keeps CLS and the floor(keep_ratio * N) patch
 * tokens with the highest scores (ties to the lower position), in order.
 * Exit (exit_logits != NULL): device fp32 [batch][classes] head logits;
 * c = max softmax; a sample with delta < 1 and c >= delta leaves the batch,
 * its logits are copied to logits[i] (device fp32 [batch][classes]) and
 * exit_block[i] (device int32 [batch]) is set to 1.  Optional LayerNorm of
 * every kept row (eps 1e-6; ln_g, ln_b device fp32 [d]) into ln_out
 * (device [M][d], row j of the packed output; bf16 for precision 1, else
 * fp32).  Synchronises the stream. */
FUSION_API int fusion_test_topk_compact(const fusion_ragged* in, const float* scores, int heads,
                                        int tmax, const float* prune_w, const float* prune_b,
                                        double keep_ratio, const float* exit_logits,
                                        int classes, float delta, float* logits,
                                        int32_t* exit_block, int precision, const float* ln_g,
                                        const float* ln_b, void* ln_out,
                                        const fusion_packed_out* out, void* stream);

/* Message of the last failed call on this thread ("" if none). */
FUSION_API const char* fusion_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FUSION_H */
