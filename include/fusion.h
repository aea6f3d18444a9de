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
 * 2^31 (the residual stream's element count).  *out receives the handle.
 * Errors: FUSION_E_INVALID_ARG, FUSION_E_BLOB (before any device call),
 * FUSION_E_CAPACITY (max_batch beyond the residual-stream limit),
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
 * pruning.  Range [0, 16].  Errors: FUSION_E_INVALID_ARG. */
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

/* Message of the last failed call on this thread ("" if none). */
FUSION_API const char* fusion_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* FUSION_H */
