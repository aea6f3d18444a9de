// Kernel-level entry points of the C ABI: each runs the kernels that
// fusion_run launches for one step of Algorithm 1 (Sec. III-B..E), on
// caller-supplied packed ragged buffers instead of the model's workspace, so
// that a step can be checked, or used, on its own.  Host arrays describe the
// ragged layout (per-sample offsets, merge counts); every argument is checked
// on the host before anything is enqueued.  The calls that need scratch
// (identity live and row maps, device copies of the offsets, keep flags)
// allocate it for the call and synchronise the stream before freeing it.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <mutex>
#include <string>

#include "../../include/fusion.h"
#include "kernels.h"

using namespace fusion;

// Scratch of fusion_test_merge_noalloc: a static device array, one copy per
// GPU the library runs on, held until the process ends.  Host code never
// passes the array's name to a kernel (on the host it is a stand-in, not a
// device address): its address on the current device comes from
// hipGetSymbolAddress, looked up once per device.
constexpr size_t kNoAllocScratchBytes = (size_t)1 << 20;
static __device__ __align__(256) char scratch[kNoAllocScratchBytes];

namespace {

int bad(const std::string& m) { return api_fail(FUSION_E_INVALID_ARG, m.c_str()); }

int hip_fail(const char* what, hipError_t e) {
  return api_fail(FUSION_E_HIP, (std::string(what) + ": " + hipGetErrorString(e)).c_str());
}

#define HIP_TRY(expr)                               \
  do {                                              \
    hipError_t e_ = (expr);                         \
    if (e_ != hipSuccess) return hip_fail(#expr, e_); \
  } while (0)

constexpr int kMaxTokens = 640;  // tokens per sample, the adapt / attention limit

// Offsets of a packed ragged batch (host): cu[0] = 0, every sample holds
// 1 .. kMaxTokens rows.  Returns the row count and the largest sample.
int check_offsets(const int32_t* cu, int batch, int* M, int* T_ub) {
  if (!cu) return bad("offsets are null");
  if (batch < 1 || batch > 65536) return bad("batch must be in 1 .. 65536");
  if (cu[0] != 0) return bad("offsets must start at 0");
  int tmax = 0;
  for (int i = 0; i < batch; i++) {
    const long t = (long)cu[i + 1] - cu[i];
    if (t < 1 || t > kMaxTokens)
      return bad("sample " + std::to_string(i) + " has " + std::to_string(t) +
                 " rows (1 .. 640 allowed)");
    tmax = std::max(tmax, (int)t);
  }
  // row offsets into the fp32 rows are 32-bit in the adapt kernel
  if ((long)cu[batch] * 768 > (long)INT32_MAX) return bad("too many rows");
  *M = cu[batch];
  *T_ub = tmax;
  return FUSION_OK;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Scratch of one adaptive-step call, carved from one device buffer.
struct StepScratch {
  int* cu;          // [B + 1]
  int* live;        // [B] identity
  int* rmap;        // [M] identity
  float* size;      // [M] working copy (the merge adds sizes in place)
  int* keep;        // [M]
  int* newlen;      // [B]
  int* r;           // [B]
  LiveCounts* cnt;  // nlive = B, M
  float* sim_v;     // [B][AD_SIM_STRIDE] best matches of long samples
  int* sim_i;
};

// with_sim: also the best-match buffers that let long samples spread the
// merge similarity over several workgroups (results are identical without)
size_t step_scratch_bytes(int B, int M, bool with_sim = false) {
  return align256((size_t)(B + 1) * 4) + 3 * align256((size_t)B * 4) +
         3 * align256((size_t)M * 4) + align256(sizeof(LiveCounts)) +
         (with_sim ? 2 * align256((size_t)B * AD_SIM_STRIDE * 4) : 0);
}

StepScratch carve(char* p, int B, int M, bool with_sim = false) {
  StepScratch s;
  auto take = [&](size_t bytes) {
    char* q = p;
    p += align256(bytes);
    return q;
  };
  s.cu = (int*)take((size_t)(B + 1) * 4);
  s.live = (int*)take((size_t)B * 4);
  s.newlen = (int*)take((size_t)B * 4);
  s.r = (int*)take((size_t)B * 4);
  s.rmap = (int*)take((size_t)M * 4);
  s.size = (float*)take((size_t)M * 4);
  s.keep = (int*)take((size_t)M * 4);
  s.cnt = (LiveCounts*)take(sizeof(LiveCounts));
  s.sim_v = with_sim ? (float*)take((size_t)B * AD_SIM_STRIDE * 4) : nullptr;
  s.sim_i = with_sim ? (int*)take((size_t)B * AD_SIM_STRIDE * 4) : nullptr;
  return s;
}

// Per-call device scratch: allocated here, freed after the stream has
// drained (the kernels read it until then).
struct CallScratch {
  char* p = nullptr;
  hipStream_t s;
  explicit CallScratch(hipStream_t s_) : s(s_) {}
  hipError_t alloc(size_t bytes) { return hipMalloc((void**)&p, bytes); }
  ~CallScratch() {
    if (p) {
      hipStreamSynchronize(s);
      hipFree(p);
    }
  }
};

int check_ragged(const fusion_ragged* in, int* M, int* T_ub) {
  if (!in) return bad("ragged input is null");
  if (!in->x || !in->size || !in->origin) return bad("null row buffer");
  if (in->d < 32 || in->d > 768 || in->d % 32) return bad("width d must be a multiple of 32 in 32 .. 768");
  return check_offsets(in->cu, in->batch, M, T_ub);
}

int check_packed_out(const fusion_packed_out* o) {
  if (!o) return bad("packed output is null");
  if (!o->rows || !o->size || !o->origin || !o->cu || !o->live || !o->counts)
    return bad("null packed output buffer");
  return FUSION_OK;
}

// Copy the offsets (and merge counts) to the scratch, the working sizes,
// and set the identity maps.
int prepare(const fusion_ragged* in, const int32_t* r, int M, StepScratch& sc, hipStream_t s) {
  const int B = in->batch;
  HIP_TRY(hipMemcpyAsync(sc.cu, in->cu, (size_t)(B + 1) * 4, hipMemcpyHostToDevice, s));
  if (r) HIP_TRY(hipMemcpyAsync(sc.r, r, (size_t)B * 4, hipMemcpyHostToDevice, s));
  HIP_TRY(hipMemcpyAsync(sc.size, in->size, (size_t)M * 4, hipMemcpyDeviceToDevice, s));
  HIP_TRY(launch_step_init(sc.live, B, sc.rmap, M, sc.cnt, s));
  return FUSION_OK;
}

template <typename T>
int compact(const fusion_ragged* in, const StepScratch& sc, int T_ub,
            const float* ln_g, const float* ln_b, void* ln_out,
            const fusion_packed_out* o, hipStream_t s) {
  CompactArgs c{};
  c.x = in->x; c.rmap = sc.rmap; c.size = sc.size; c.origin = in->origin;
  c.cu = sc.cu; c.live = sc.live; c.cnt = sc.cnt; c.keep = sc.keep; c.newlen = sc.newlen;
  c.rmap2 = o->rows; c.size2 = o->size; c.origin2 = o->origin; c.cu2 = o->cu;
  c.live2 = o->live; c.cnt2 = (LiveCounts*)o->counts;
  c.d = in->d; c.n0 = T_ub - 1; c.B = in->batch; c.b = 1; c.tr_ids = nullptr;
  c.nlive_ub = in->batch;
  c.ln_g = ln_g; c.ln_b = ln_b; c.ln_out = ln_out;
  HIP_TRY(launch_compact<T>(c, s));
  return FUSION_OK;
}

int merge_impl(const fusion_ragged* in, const int32_t* r, int id_stride, int32_t* merge_dst,
               const fusion_packed_out* out, hipStream_t s, char* mem, size_t mem_cap,
               int* M_out, bool with_sim) {
  int M = 0, T_ub = 0;
  if (int rc = check_ragged(in, &M, &T_ub)) return rc;
  if (int rc = check_packed_out(out)) return rc;
  if (!r) return bad("merge counts are null");
  for (int i = 0; i < in->batch; i++) {
    const int N = in->cu[i + 1] - in->cu[i] - 1;
    if (r[i] < 0 || r[i] > N / 2)
      return bad("merge count of sample " + std::to_string(i) + " outside 0 .. floor(N/2)");
  }
  if (merge_dst && (id_stride < 1 || id_stride > (1 << 20))) return bad("id_stride out of range");
  *M_out = M;
  if (!mem) return FUSION_OK;  // sizing pass
  if (step_scratch_bytes(in->batch, M, with_sim) > mem_cap) return bad("scratch too small");
  StepScratch sc = carve(mem, in->batch, M, with_sim);
  if (int rc = prepare(in, r, M, sc, s)) return rc;
  AdaptArgs a{};
  a.x = in->x; a.rmap = sc.rmap; a.size = sc.size; a.origin = in->origin;
  a.cu = sc.cu; a.live = sc.live; a.cnt = sc.cnt;
  a.d = in->d; a.H = 1; a.n0 = merge_dst ? id_stride - 1 : T_ub - 1; a.C = 0; a.L = 1;
  a.B = in->batch; a.b = 1;
  a.isM = 1; a.isE = 0; a.isP = 0;
  a.r_fixed = sc.r; a.rho = 1.0; a.delta = 1.0f; a.tau_eff = 1.0;
  a.tmax = T_ub; a.keep = sc.keep; a.newlen = sc.newlen;
  a.tr_merge = merge_dst;
  a.sim_v = sc.sim_v; a.sim_i = sc.sim_i;
  a.nlive_ub = in->batch; a.T_ub = T_ub;
  HIP_TRY(launch_adapt(a, s));
  return compact<float>(in, sc, T_ub, nullptr, nullptr, nullptr, out, s);
}

// Device address of `scratch` on the current device, looked up on the
// first call on each device (with that device current) and kept.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
char* g_scratch_ptr[kMaxDevices] = {};

int noalloc_scratch(char** out) {
  int dev = 0;
  HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return bad("device index beyond the scratch table");
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    HIP_TRY(hipGetSymbolAddress((void**)&ptr, HIP_SYMBOL(scratch)));
    if (!ptr) return api_fail(FUSION_E_HIP, "no device address for the static scratch");
    g_scratch_ptr[dev] = (char*)ptr;
  }
  *out = g_scratch_ptr[dev];
  return FUSION_OK;
}

}  // namespace

extern "C" {

FUSION_API int fusion_test_gemm(int precision, const void* A, int lda, const void* W, int N,
                                int K, int M, const float* bias, int epi, void* out, int ldo,
                                const int32_t* rows, void* stream) {
  if (precision != 0 && precision != 1) return bad("precision must be 0 (fp32) or 1 (bf16)");
  if (!A || !W || !bias || !out) return bad("null buffer");
  if (M < 1 || N < 4 || K < 1) return bad("M >= 1, N >= 4 and K >= 1 required");
  if (epi < FUSION_EPI_STORE || epi > FUSION_EPI_F32) return bad("unknown epilogue");
  if (lda < K || ldo < N) return bad("leading dimensions below K / N");
  if (rows && (epi == FUSION_EPI_STORE || epi == FUSION_EPI_GELU))
    return bad("a row map applies to the fp32 epilogues only");
  if (precision == 1) {
    if (K % 32 || lda % 8) return bad("bf16 GEMM needs K % 32 == 0 and lda % 8 == 0");
    if (N % 4 || ldo % 4) return bad("bf16 GEMM needs N and ldo multiples of 4");
    if ((epi == FUSION_EPI_STORE || epi == FUSION_EPI_GELU) && (N % 8 || ldo % 8))
      return bad("bf16 outputs need N and ldo multiples of 8");
  }
  const int mode = epi == FUSION_EPI_STORE ? EPI_STORE
                   : epi == FUSION_EPI_GELU ? EPI_GELU
                   : epi == FUSION_EPI_RESID ? EPI_RESID : EPI_F32;
  Epi e{mode, out, ldo, bias, rows, nullptr, 0};
  hipStream_t s = (hipStream_t)stream;
  hipError_t err =
      precision == 1
          ? launch_gemm<bf16_t>((const bf16_t*)A, lda, (const bf16_t*)W, N, K, nullptr, M, M, e, s)
          : launch_gemm<float>((const float*)A, lda, (const float*)W, N, K, nullptr, M, M, e, s);
  if (err != hipSuccess) return hip_fail("launch_gemm", err);
  return FUSION_OK;
}

FUSION_API int fusion_test_attention(int precision, const void* qkv, const float* size,
                                     const int32_t* cu, int batch, int heads, int d,
                                     int prop_attn, void* out, float* cls_scores, int tmax,
                                     void* stream) {
  if (precision != 0 && precision != 1) return bad("precision must be 0 (fp32) or 1 (bf16)");
  if (!qkv || !size || !out) return bad("null buffer");
  if (heads < 1 || d < 1 || d % heads || d % 4 || d > 768) return bad("bad width or heads");
  if (prop_attn != 0 && prop_attn != 1) return bad("prop_attn must be 0 or 1");
  int M = 0, T_ub = 0;
  if (int rc = check_offsets(cu, batch, &M, &T_ub)) return rc;
  if (cls_scores && tmax < T_ub) return bad("tmax below the longest sample");
  const int dh = d / heads;
  if (precision == 1 && dh != 64) return bad("the bf16 attention kernels need 64-wide heads");
  hipStream_t s = (hipStream_t)stream;
  CallScratch mem(s);
  HIP_TRY(mem.alloc(step_scratch_bytes(batch, M)));
  StepScratch sc = carve(mem.p, batch, M);
  HIP_TRY(hipMemcpyAsync(sc.cu, cu, (size_t)(batch + 1) * 4, hipMemcpyHostToDevice, s));
  HIP_TRY(launch_step_init(sc.live, batch, sc.rmap, M, sc.cnt, s));
  AttnArgs a{};
  a.qkv = qkv; a.size = size; a.cu = sc.cu; a.live = sc.live; a.cnt = sc.cnt;
  a.H = heads; a.dh = dh; a.d = d; a.scale = (float)(1.0 / std::sqrt((double)dh));
  a.prop_attn = prop_attn; a.out = out; a.cls_scores = cls_scores; a.tmax = tmax;
  a.token_counts = nullptr; a.L = 1; a.b0 = 0; a.nlive_ub = batch; a.T_ub = T_ub;
  hipError_t err = precision == 1 ? launch_attention<bf16_t>(a, s) : launch_attention<float>(a, s);
  if (err != hipSuccess) return hip_fail("launch_attention", err);
  return FUSION_OK;
}

FUSION_API int fusion_test_merge(const fusion_ragged* in, const int32_t* r, int id_stride,
                                 int32_t* merge_dst, const fusion_packed_out* out,
                                 void* stream) {
  hipStream_t s = (hipStream_t)stream;
  int M = 0;
  if (int rc = merge_impl(in, r, id_stride, merge_dst, out, s, nullptr, 0, &M, true)) return rc;
  CallScratch mem(s);
  const size_t need = step_scratch_bytes(in->batch, M, true);
  HIP_TRY(mem.alloc(need));
  return merge_impl(in, r, id_stride, merge_dst, out, s, mem.p, need, &M, true);
}

FUSION_API int fusion_test_merge_noalloc(const fusion_ragged* in, const int32_t* r,
                                         int id_stride, int32_t* merge_dst,
                                         const fusion_packed_out* out, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  int M = 0;
  if (int rc = merge_impl(in, r, id_stride, merge_dst, out, s, nullptr, 0, &M, false)) return rc;
  const size_t need = step_scratch_bytes(in->batch, M);
  if (need > kNoAllocScratchBytes)
    return api_fail(FUSION_E_CAPACITY,
                    ("the call needs " + std::to_string(need) + " bytes of scratch; the static " +
                     "array holds " + std::to_string(kNoAllocScratchBytes))
                        .c_str());
  char* mem = nullptr;
  if (int rc = noalloc_scratch(&mem)) return rc;
  // every scratch word the kernels read is written earlier in this call
  // (offsets, counts and sizes copied in, maps set by the init kernel, keep
  // flags and new lengths by the adapt kernel), so nothing is cleared
  return merge_impl(in, r, id_stride, merge_dst, out, s, mem, kNoAllocScratchBytes, &M, false);
}

FUSION_API int fusion_test_topk_compact(const fusion_ragged* in, const float* scores, int heads,
                                        int tmax, const float* prune_w, const float* prune_b,
                                        double keep_ratio, const float* exit_logits,
                                        int classes, float delta, float* logits,
                                        int32_t* exit_block, int precision, const float* ln_g,
                                        const float* ln_b, void* ln_out,
                                        const fusion_packed_out* out, void* stream) {
  int M = 0, T_ub = 0;
  if (int rc = check_ragged(in, &M, &T_ub)) return rc;
  if (int rc = check_packed_out(out)) return rc;
  if (!scores && !(prune_w && prune_b)) return bad("give CLS-attention scores or a learned scorer");
  if (scores && (heads < 1 || heads > 64 || tmax < T_ub)) return bad("bad score layout");
  if (!(keep_ratio >= 0.0 && keep_ratio <= 1.0)) return bad("keep ratio outside [0, 1]");
  if (exit_logits) {
    if (classes < 1 || !logits || !exit_block) return bad("exit check needs classes, logits and exit_block");
    if (!(delta >= 0.f && delta <= 1.f)) return bad("threshold outside [0, 1]");
  }
  if (precision != 0 && precision != 1) return bad("precision must be 0 (fp32) or 1 (bf16)");
  if (ln_out && (!ln_g || !ln_b)) return bad("LayerNorm output needs its gain and bias");
  hipStream_t s = (hipStream_t)stream;
  CallScratch mem(s);
  HIP_TRY(mem.alloc(step_scratch_bytes(in->batch, M)));
  StepScratch sc = carve(mem.p, in->batch, M);
  if (int rc = prepare(in, nullptr, M, sc, s)) return rc;
  AdaptArgs a{};
  a.x = in->x; a.rmap = sc.rmap; a.size = sc.size; a.origin = in->origin;
  a.cu = sc.cu; a.live = sc.live; a.cnt = sc.cnt;
  a.d = in->d; a.H = scores ? heads : 1; a.n0 = T_ub - 1; a.C = exit_logits ? classes : 0;
  a.L = 1; a.B = in->batch; a.b = 1;
  a.isM = 0; a.isE = exit_logits ? 1 : 0; a.isP = 1;
  a.prune_rule = scores ? FUSION_PRUNE_CLS_ATTN : FUSION_PRUNE_LEARNED;
  a.prune_w = prune_w; a.prune_b = prune_b;
  a.head_buf = exit_logits; a.delta = exit_logits ? delta : 1.0f;
  a.logits = logits; a.exit_block = exit_block;
  a.cls_scores = scores; a.tmax = tmax; a.tau_eff = keep_ratio;
  a.keep = sc.keep; a.newlen = sc.newlen;
  a.nlive_ub = in->batch; a.T_ub = T_ub;
  HIP_TRY(launch_adapt(a, s));
  if (precision == 1) return compact<bf16_t>(in, sc, T_ub, ln_g, ln_b, ln_out, out, s);
  return compact<float>(in, sc, T_ub, ln_g, ln_b, ln_out, out, s);
}

}  // extern "C"
