// C ABI and host orchestration of Fusion's staged adaptive ViT inference.
//
// fusion_run enqueues Algorithm 1 (Sec. III-B) for a whole batch on one
// stream without any host synchronisation: live-sample and token counts stay
// on the device (LiveCounts), and every grid is sized for a host-side upper
// bound (tiles or samples beyond the live count return at once).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <string>
#include <vector>

#include "../../include/fusion.h"
#include "kernels.h"

using namespace fusion;

namespace {

thread_local std::string g_err;

int fail(int code, const std::string& msg) {
  g_err = msg;
  return code;
}

#define HIP_OR_FAIL(expr)                                                   \
  do {                                                                      \
    hipError_t e_ = (expr);                                                 \
    if (e_ != hipSuccess)                                                   \
      return fail(FUSION_E_HIP, std::string(#expr) + ": " + hipGetErrorString(e_)); \
  } while (0)

// ----------------------------------------------------------- blob format --
constexpr char kMagic[8] = {'F', 'U', 'S', 'N', 'V', 'I', 'T', '\0'};
constexpr uint32_t kVersion = 2;
constexpr size_t kHeaderBytes = 724;  // see the blob writer's layout
constexpr size_t kEntryBytes = 68;

struct TensorRef {
  std::string name;
  std::vector<int64_t> shape;
  uint64_t offset = 0, nbytes = 0;
};

struct Config {
  int img, patch, in_ch, d, heads, L, mlp, C;
  int prop_attn, precision;
  uint32_t merge_mask, exit_mask, prune_mask;
  int r_b[FUSION_MAX_LAYERS];
  double tau_b[FUSION_MAX_LAYERS];
  float delta_b[FUSION_MAX_LAYERS];
  int merge_rule, prune_rule;            // FUSION_MERGE_*, FUSION_PRUNE_*
  int exit_kind[FUSION_MAX_LAYERS];      // FUSION_EXIT_* (exit blocks)
  int exit_hidden;
  int n0, pdim, dh;
  std::vector<int> exits;
};

template <typename V>
V rd(const uint8_t* p, size_t off) {
  V v;
  std::memcpy(&v, p + off, sizeof(V));
  return v;
}

std::vector<std::pair<std::string, std::vector<int64_t>>> expected_tensors(const Config& c) {
  std::vector<std::pair<std::string, std::vector<int64_t>>> v;
  const int64_t d = c.d, mlp = c.mlp, C = c.C;
  v.push_back({"cls", {d}});
  v.push_back({"pos", {c.n0 + 1, d}});
  v.push_back({"pe_w", {d, c.pdim}});
  v.push_back({"pe_b", {d}});
  for (int b = 1; b <= c.L; b++) {
    const std::string p = "blk" + std::to_string(b) + ".";
    v.push_back({p + "ln1_g", {d}});
    v.push_back({p + "ln1_b", {d}});
    v.push_back({p + "qkv_w", {3 * d, d}});
    v.push_back({p + "qkv_b", {3 * d}});
    v.push_back({p + "proj_w", {d, d}});
    v.push_back({p + "proj_b", {d}});
    v.push_back({p + "ln2_g", {d}});
    v.push_back({p + "ln2_b", {d}});
    v.push_back({p + "fc1_w", {mlp, d}});
    v.push_back({p + "fc1_b", {mlp}});
    v.push_back({p + "fc2_w", {d, mlp}});
    v.push_back({p + "fc2_b", {d}});
    if (c.merge_mask >> (b - 1) & 1) {
      v.push_back({p + "router_w", {d}});
      v.push_back({p + "router_b", {1}});
    }
    if (c.exit_mask >> (b - 1) & 1) {
      v.push_back({p + "eln_g", {d}});
      v.push_back({p + "eln_b", {d}});
      if (c.exit_kind[b - 1] == FUSION_EXIT_LINEAR) {
        v.push_back({p + "ew", {C, d}});
        v.push_back({p + "eb", {C}});
      } else {
        const int64_t hx = c.exit_hidden;
        v.push_back({p + "ew1", {hx, d}});
        v.push_back({p + "eb1", {hx}});
        v.push_back({p + "ew2", {C, hx}});
        v.push_back({p + "eb2", {C}});
      }
    }
    if ((c.prune_mask >> (b - 1) & 1) && c.prune_rule == FUSION_PRUNE_LEARNED) {
      v.push_back({p + "prune_w", {d}});
      v.push_back({p + "prune_b", {1}});
    }
  }
  v.push_back({"norm_g", {d}});
  v.push_back({"norm_b", {d}});
  v.push_back({"head_w", {C, d}});
  v.push_back({"head_b", {C}});
  return v;
}

int parse_blob(const void* blob, size_t bytes, Config& c,
               std::vector<TensorRef>& tensors) {
  if (!blob) return fail(FUSION_E_INVALID_ARG, "blob is null");
  if (bytes < kHeaderBytes) return fail(FUSION_E_BLOB, "blob shorter than its header");
  const uint8_t* p = (const uint8_t*)blob;
  if (std::memcmp(p, kMagic, 8) != 0) return fail(FUSION_E_BLOB, "bad magic");
  if (rd<uint32_t>(p, 8) != kVersion) return fail(FUSION_E_BLOB, "unsupported blob version");
  if (rd<uint32_t>(p, 12) != kHeaderBytes) return fail(FUSION_E_BLOB, "bad header size");
  uint32_t u[8];
  for (int k = 0; k < 8; k++) u[k] = rd<uint32_t>(p, 16 + 4 * k);
  for (int k = 0; k < 8; k++)
    if (u[k] == 0 || u[k] > (1u << 20)) return fail(FUSION_E_BLOB, "dimension out of range");
  c.img = u[0]; c.patch = u[1]; c.in_ch = u[2]; c.d = u[3];
  c.heads = u[4]; c.L = u[5]; c.mlp = u[6]; c.C = u[7];
  c.prop_attn = rd<uint32_t>(p, 48);
  c.precision = rd<uint32_t>(p, 52);
  c.merge_mask = rd<uint32_t>(p, 56);
  c.exit_mask = rd<uint32_t>(p, 60);
  c.prune_mask = rd<uint32_t>(p, 64);
  if (c.L > FUSION_MAX_LAYERS) return fail(FUSION_E_BLOB, "too many layers");
  if (c.img % c.patch) return fail(FUSION_E_BLOB, "image side not a multiple of the patch");
  if (c.d % c.heads) return fail(FUSION_E_BLOB, "width not a multiple of heads");
  if (c.prop_attn > 1 || c.precision > 1) return fail(FUSION_E_BLOB, "bad flags");
  const uint32_t lmask = c.L == 32 ? 0xffffffffu : ((1u << c.L) - 1u);
  if ((c.merge_mask | c.exit_mask | c.prune_mask) & ~lmask)
    return fail(FUSION_E_BLOB, "layer mask names a block beyond L");
  for (int b = 0; b < FUSION_MAX_LAYERS; b++) {
    c.r_b[b] = (int)rd<uint32_t>(p, 68 + 4 * b);
    c.tau_b[b] = rd<double>(p, 196 + 8 * b);
    c.delta_b[b] = rd<float>(p, 452 + 4 * b);
    if (b < c.L) {
      if (c.r_b[b] < 0 || c.r_b[b] > (1 << 20)) return fail(FUSION_E_BLOB, "bad merge budget");
      if (!(c.tau_b[b] >= 0.0 && c.tau_b[b] <= 1.0)) return fail(FUSION_E_BLOB, "bad keep ratio");
      if (!(c.delta_b[b] >= 0.f && c.delta_b[b] <= 1.f)) return fail(FUSION_E_BLOB, "bad exit threshold");
    }
  }
  c.merge_rule = (int)rd<uint32_t>(p, 580);
  c.prune_rule = (int)rd<uint32_t>(p, 584);
  if (c.merge_rule > FUSION_MERGE_FRACTION) return fail(FUSION_E_BLOB, "unknown merge rule");
  if (c.prune_rule > FUSION_PRUNE_LEARNED) return fail(FUSION_E_BLOB, "unknown prune rule");
  bool any_mlp = false;
  for (int b = 0; b < FUSION_MAX_LAYERS; b++) {
    const uint32_t k = rd<uint32_t>(p, 588 + 4 * b);
    const bool is_exit = b < c.L && (c.exit_mask >> b & 1);
    if (k > FUSION_EXIT_POOL_MLP || (k != 0 && !is_exit))
      return fail(FUSION_E_BLOB, "bad exit-head kind");
    c.exit_kind[b] = (int)k;
    any_mlp = any_mlp || k != FUSION_EXIT_LINEAR;
  }
  const uint32_t hx = rd<uint32_t>(p, 716);
  if (any_mlp && (hx == 0 || hx > 8192 || hx % (c.precision == 1 ? 64 : 32)))
    return fail(FUSION_E_BLOB, "exit hidden width must be a multiple of 64 (bf16) or 32 (fp32), at most 8192");
  c.exit_hidden = any_mlp ? (int)hx : 0;
  c.n0 = (c.img / c.patch) * (c.img / c.patch);
  c.pdim = c.in_ch * c.patch * c.patch;
  c.dh = c.d / c.heads;
  c.exits.clear();
  for (int b = 1; b <= c.L; b++)
    if (c.exit_mask >> (b - 1) & 1) c.exits.push_back(b);
  // limits of the kernels
  if (c.n0 + 1 > 640) return fail(FUSION_E_BLOB, "more than 640 tokens per sample");
  if (c.patch % 4) return fail(FUSION_E_BLOB, "patch side must be a multiple of 4");
  if (c.d > 768 || c.d % 16) return fail(FUSION_E_BLOB, "width must be a multiple of 16 and <= 768");
  if (c.precision == 1 && (c.d % 64 || c.mlp % 64 || c.pdim % 64))
    return fail(FUSION_E_BLOB, "bf16 path needs width, MLP width and patch size multiples of 64");

  const uint32_t nt = rd<uint32_t>(p, 720);
  auto exp = expected_tensors(c);
  if (nt != exp.size()) return fail(FUSION_E_BLOB, "tensor count does not match the header");
  if (kHeaderBytes + (size_t)nt * kEntryBytes > bytes) return fail(FUSION_E_BLOB, "truncated tensor table");
  tensors.clear();
  for (uint32_t k = 0; k < nt; k++) {
    const uint8_t* e = p + kHeaderBytes + (size_t)k * kEntryBytes;
    char name[33];
    std::memcpy(name, e, 32);
    name[32] = 0;
    TensorRef t;
    t.name = name;
    const uint32_t ndim = rd<uint32_t>(e, 32);
    if (ndim < 1 || ndim > 4) return fail(FUSION_E_BLOB, "bad rank for " + t.name);
    int64_t count = 1;
    for (uint32_t q = 0; q < ndim; q++) {
      t.shape.push_back(rd<uint32_t>(e, 36 + 4 * q));
      count *= t.shape.back();
    }
    t.offset = rd<uint64_t>(e, 52);
    t.nbytes = rd<uint64_t>(e, 60);
    if (t.name != exp[k].first) return fail(FUSION_E_BLOB, "expected tensor " + exp[k].first + ", found " + t.name);
    if (t.shape != exp[k].second) return fail(FUSION_E_BLOB, "wrong shape for " + t.name);
    if (t.nbytes != (uint64_t)count * 4) return fail(FUSION_E_BLOB, "wrong byte size for " + t.name);
    if (t.offset % 4 || t.offset < kHeaderBytes || t.offset > bytes || t.nbytes > bytes - t.offset)
      return fail(FUSION_E_BLOB, "tensor " + t.name + " outside the blob");
    tensors.push_back(t);
  }
  return FUSION_OK;
}

void fill_info(const Config& c, fusion_info* o) {
  std::memset(o, 0, sizeof(*o));
  o->img = c.img; o->patch = c.patch; o->in_ch = c.in_ch; o->d = c.d;
  o->heads = c.heads; o->layers = c.L; o->mlp = c.mlp; o->classes = c.C;
  o->n0 = c.n0; o->precision = c.precision; o->prop_attn = c.prop_attn;
  o->merge_mask = c.merge_mask; o->exit_mask = c.exit_mask; o->prune_mask = c.prune_mask;
  o->n_exit = (int)c.exits.size();
  for (int k = 0; k < o->n_exit; k++) {
    o->exit_blocks[k] = c.exits[k];
    o->delta[k] = c.delta_b[c.exits[k] - 1];
  }
  for (int b = 0; b < FUSION_MAX_LAYERS; b++) {
    o->r_b[b] = c.r_b[b];
    o->tau_b[b] = c.tau_b[b];
    o->exit_kind[b] = c.exit_kind[b];
  }
  o->rho = 1.0;
  o->merge_rule = c.merge_rule;
  o->prune_rule = c.prune_rule;
  o->exit_hidden = c.exit_hidden;
}

uint16_t host_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

// ------------------------------------------------------------ profiling --
enum Kind {
  K_INIT, K_PATCH, K_LN, K_QKV, K_ATTN, K_PROJ, K_FC1, K_FC2, K_EXIT_HEAD,
  K_ADAPT, K_COMPACT, K_FINAL_HEAD, K_COUNT
};
const char* kKindNames[K_COUNT] = {
    "init", "patch_embed", "layernorm", "gemm_qkv", "attention", "gemm_proj",
    "gemm_fc1_gelu", "gemm_fc2", "exit_head", "adapt", "compact", "final_head"};

}  // namespace

int fusion::api_fail(int code, const char* msg) { return fail(code, msg); }

struct BlockW {
  const float *ln1_g, *ln1_b, *qkv_b, *proj_b, *ln2_g, *ln2_b, *fc1_b, *fc2_b;
  const void *qkv_w, *proj_w, *fc1_w, *fc2_w;
  const float *router_w, *router_b, *eln_g, *eln_b, *eb;
  const void* ew;
  // MLP exit heads (FUSION_EXIT_CLS_MLP / POOL_MLP) and the learned scorer
  const float *eb1, *eb2, *prune_w, *prune_b;
  const void *ew1, *ew2;
};

struct fusion_model {
  Config cfg;
  int max_batch = 0;
  int device = 0;
  std::vector<void*> allocs;
  // weights
  float* wf32 = nullptr;  // the blob's tensor data, fp32
  void* wmat = nullptr;   // matrix weights in the compute type (bf16 path)
  const float *cls, *pos, *pe_b, *norm_g, *norm_b, *head_b;
  const void *pe_w, *head_w;
  BlockW blk[FUSION_MAX_LAYERS];
  // workspace
  float* x;        // [Mmax, d] fp32 residual stream; rows never move
  int* rmap[2];    // packed row -> physical row of x (ping-pong)
  float* size[2];
  int* origin[2];
  int* cu[2];
  int* live[2];
  LiveCounts* cnt[2];
  void* act;   // [Mmax, d]
  void* qkv;   // [Mmax, 3d]
  void* ffn;   // [Mmax, mlp] (also the patch matrix)
  void* hc;    // [max_batch, d]
  void* hbuf;  // [max_batch, exit_hidden] (MLP exit heads)
  float* head_buf;
  float* cls_scores;
  int* keep;
  int* newlen;
  float* sim_v;  // [max_batch][AD_SIM_STRIDE] best-match similarities (long samples)
  int* sim_i;
  // runtime parameters
  float delta[FUSION_MAX_LAYERS];  // per exit head
  double rho = 1.0;
  // profiling
  bool prof = false;
  struct Rec { int kind; hipEvent_t a, b; };
  std::vector<Rec> recs;
  std::vector<hipEvent_t> pool;
  double tot_ms[K_COUNT] = {};
  int64_t launches[K_COUNT] = {};
};

namespace {

template <typename T>
void* dev_alloc(fusion_model* m, size_t bytes, int* rc) {
  void* p = nullptr;
  if (bytes == 0) bytes = 256;
  if (hipMalloc(&p, bytes) != hipSuccess) {
    *rc = fail(FUSION_E_OOM, "hipMalloc of " + std::to_string(bytes) + " bytes failed");
    return nullptr;
  }
  m->allocs.push_back(p);
  return p;
}

hipEvent_t get_event(fusion_model* m) {
  if (!m->pool.empty()) {
    hipEvent_t e = m->pool.back();
    m->pool.pop_back();
    return e;
  }
  hipEvent_t e;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

struct Prof {
  fusion_model* m;
  hipStream_t s;
  int kind;
  hipEvent_t a = nullptr;
  Prof(fusion_model* m_, hipStream_t s_, int k) : m(m_), s(s_), kind(k) {
    if (m->prof) {
      a = get_event(m);
      if (a) hipEventRecord(a, s);
    }
  }
  ~Prof() {
    if (m->prof && a) {
      hipEvent_t b = get_event(m);
      if (b) {
        hipEventRecord(b, s);
        m->recs.push_back({kind, a, b});
      }
    }
  }
};

void release_all(fusion_model* m) {
  for (void* p : m->allocs) hipFree(p);
  m->allocs.clear();
  for (auto& r : m->recs) {
    hipEventDestroy(r.a);
    hipEventDestroy(r.b);
  }
  m->recs.clear();
  for (auto e : m->pool) hipEventDestroy(e);
  m->pool.clear();
}

struct RunOpts {
  const fusion_trace* trace = nullptr;
  int stop_block = 0;  // debug: 0 = full run
  int stop_stage = 0;
};

template <typename T>
int run_impl(fusion_model* m, const float* images, int B, float* logits,
             int32_t* exit_block, int32_t* token_counts, const RunOpts& o,
             hipStream_t s, int* cur_out) {
  const Config& c = m->cfg;
  const int d = c.d, n0 = c.n0, T0 = n0 + 1, L = c.L;
  int cur = 0;
  {
    Prof p(m, s, K_INIT);
    HIP_OR_FAIL(launch_init(m->x, m->rmap[0], m->size[0], m->origin[0], m->cu[0], m->live[0],
                            m->cnt[0], token_counts, m->cls, m->pos, B, n0, d, L, s));
  }
  {
    Prof p(m, s, K_PATCH);
    HIP_OR_FAIL(launch_patchify<T>(images, (T*)m->ffn, B, c.in_ch, c.img, c.patch, s));
    Epi e{EPI_PATCH, m->x, d, m->pe_b, nullptr, m->pos, n0};
    HIP_OR_FAIL(launch_gemm<T>((const T*)m->ffn, c.pdim, (const T*)m->pe_w, d, c.pdim,
                               nullptr, B * n0, B * n0, e, s));
  }
  if (o.stop_block > 0 && o.stop_stage == 0) {
    *cur_out = cur;
    return FUSION_OK;
  }
  const float scale = (float)(1.0 / std::sqrt((double)c.dh));
  const double tau_rho = m->rho;
  int T_ub = T0;
  const fusion_trace* tr = o.trace;
  bool ln1_done = false;  // act already holds this block's LN1 (from the compaction)
  for (int b = 1; b <= L; b++) {
    const BlockW& w = m->blk[b - 1];
    const bool isM = c.merge_mask >> (b - 1) & 1, isE = c.exit_mask >> (b - 1) & 1,
               isP = c.prune_mask >> (b - 1) & 1;
    const int M_ub = B * T_ub;
    const int* Mdev = &m->cnt[cur]->M;
    if (!ln1_done) {
      Prof p(m, s, K_LN);
      HIP_OR_FAIL(launch_layernorm<T>(m->x, m->rmap[cur], w.ln1_g, w.ln1_b, (T*)m->act, d, m->cnt[cur],
                                      m->cu[cur], m->live[cur], 0, M_ub, nullptr, L, s));
    }
    ln1_done = false;
    {
      Prof p(m, s, K_QKV);
      Epi e{EPI_STORE, m->qkv, 3 * d, w.qkv_b, nullptr, nullptr, 0};
      HIP_OR_FAIL(launch_gemm<T>((const T*)m->act, d, (const T*)w.qkv_w, 3 * d, d, Mdev, 0,
                                 M_ub, e, s));
    }
    {
      Prof p(m, s, K_ATTN);
      AttnArgs a{};
      a.qkv = m->qkv; a.size = m->size[cur]; a.cu = m->cu[cur]; a.live = m->live[cur];
      a.cnt = m->cnt[cur]; a.H = c.heads; a.dh = c.dh; a.d = d; a.scale = scale;
      a.prop_attn = c.prop_attn; a.out = m->act;
      a.cls_scores = isP && c.prune_rule == FUSION_PRUNE_CLS_ATTN ? m->cls_scores : nullptr;
      a.tmax = T0;
      a.token_counts = token_counts; a.L = L; a.b0 = b - 1;
      a.nlive_ub = B; a.T_ub = T_ub;
      HIP_OR_FAIL(launch_attention<T>(a, s));
    }
    {
      Prof p(m, s, K_PROJ);
      Epi e{EPI_RESID, m->x, d, w.proj_b, m->rmap[cur], nullptr, 0};
      HIP_OR_FAIL(launch_gemm<T>((const T*)m->act, d, (const T*)w.proj_w, d, d, Mdev, 0, M_ub, e, s));
    }
    if (o.stop_block == b && o.stop_stage == 1) break;
    {
      Prof p(m, s, K_LN);
      HIP_OR_FAIL(launch_layernorm<T>(m->x, m->rmap[cur], w.ln2_g, w.ln2_b, (T*)m->act, d, m->cnt[cur],
                                      m->cu[cur], m->live[cur], 0, M_ub, nullptr, L, s));
    }
    {
      Prof p(m, s, K_FC1);
      Epi e{EPI_GELU, m->ffn, c.mlp, w.fc1_b, nullptr, nullptr, 0};
      HIP_OR_FAIL(launch_gemm<T>((const T*)m->act, d, (const T*)w.fc1_w, c.mlp, d, Mdev, 0, M_ub, e, s));
    }
    {
      Prof p(m, s, K_FC2);
      Epi e{EPI_RESID, m->x, d, w.fc2_b, m->rmap[cur], nullptr, 0};
      HIP_OR_FAIL(launch_gemm<T>((const T*)m->ffn, c.mlp, (const T*)w.fc2_w, d, c.mlp, Mdev, 0,
                                 M_ub, e, s));
    }
    if (o.stop_block == b && o.stop_stage == 2) break;
    if (isE) {
      // head_b of Eq. 6 on the state before this block's merge: the CLS row
      // is untouched by merging and the size-weighted pool is invariant
      // under it, so the logits equal those after the merge
      Prof p(m, s, K_EXIT_HEAD);
      const int kind = c.exit_kind[b - 1];
      const int* nl = &m->cnt[cur]->nlive;
      if (kind == FUSION_EXIT_POOL_MLP)
        HIP_OR_FAIL(launch_pool_ln<T>(m->x, m->rmap[cur], m->size[cur], m->cu[cur], m->cnt[cur], w.eln_g,
                                      w.eln_b, (T*)m->hc, d, B, s));
      else
        HIP_OR_FAIL(launch_layernorm<T>(m->x, m->rmap[cur], w.eln_g, w.eln_b, (T*)m->hc, d, m->cnt[cur],
                                        m->cu[cur], m->live[cur], 1, B, nullptr, L, s));
      if (kind == FUSION_EXIT_LINEAR) {
        Epi e{EPI_F32, m->head_buf, c.C, w.eb, nullptr, nullptr, 0};
        HIP_OR_FAIL(launch_gemm<T>((const T*)m->hc, d, (const T*)w.ew, c.C, d, nl, 0, B, e, s));
      } else {
        const int hx = c.exit_hidden;
        Epi e1{EPI_GELU, m->hbuf, hx, w.eb1, nullptr, nullptr, 0};
        HIP_OR_FAIL(launch_gemm<T>((const T*)m->hc, d, (const T*)w.ew1, hx, d, nl, 0, B, e1, s));
        Epi e2{EPI_F32, m->head_buf, c.C, w.eb2, nullptr, nullptr, 0};
        HIP_OR_FAIL(launch_gemm<T>((const T*)m->hbuf, hx, (const T*)w.ew2, c.C, hx, nl, 0, B, e2, s));
      }
    }
    if (isM || isE || isP) {
      int exit_idx = 0;
      for (size_t k = 0; k < c.exits.size(); k++)
        if (c.exits[k] == b) exit_idx = (int)k;
      const double tau_eff = std::min(1.0, std::max(0.0, 1.0 - tau_rho * (1.0 - c.tau_b[b - 1])));
      {
        Prof p(m, s, K_ADAPT);
        AdaptArgs a{};
        a.x = m->x; a.rmap = m->rmap[cur]; a.size = m->size[cur]; a.origin = m->origin[cur];
        a.cu = m->cu[cur]; a.live = m->live[cur]; a.cnt = m->cnt[cur];
        a.d = d; a.H = c.heads; a.n0 = n0; a.C = c.C; a.L = L; a.B = B; a.b = b;
        a.isM = isM; a.isE = isE; a.isP = isP;
        a.merge_rule = c.merge_rule; a.prune_rule = c.prune_rule;
        a.prune_w = w.prune_w; a.prune_b = w.prune_b;
        a.router_w = w.router_w; a.router_b = w.router_b; a.r_b = c.r_b[b - 1]; a.rho = m->rho;
        a.head_buf = m->head_buf; a.delta = isE ? m->delta[exit_idx] : 1.0f;
        a.logits = logits; a.exit_block = exit_block;
        a.cls_scores = m->cls_scores; a.tmax = T0; a.tau_eff = tau_eff;
        a.keep = m->keep; a.newlen = m->newlen;
        a.sim_v = m->sim_v; a.sim_i = m->sim_i;
        a.tr_r = tr ? tr->r : nullptr; a.tr_m = tr ? tr->m : nullptr;
        a.tr_c = tr ? tr->c : nullptr; a.tr_merge = tr ? tr->merge_dst : nullptr;
        a.nlive_ub = B; a.T_ub = T_ub;
        HIP_OR_FAIL(launch_adapt(a, s));
      }
      {
        Prof p(m, s, K_COMPACT);
        const int nx = cur ^ 1;
        CompactArgs a{};
        a.x = m->x; a.rmap = m->rmap[cur]; a.size = m->size[cur]; a.origin = m->origin[cur];
        a.cu = m->cu[cur]; a.live = m->live[cur]; a.cnt = m->cnt[cur]; a.keep = m->keep;
        a.newlen = m->newlen;
        a.rmap2 = m->rmap[nx]; a.size2 = m->size[nx]; a.origin2 = m->origin[nx]; a.cu2 = m->cu[nx];
        a.live2 = m->live[nx]; a.cnt2 = m->cnt[nx];
        a.d = d; a.n0 = n0; a.B = B; a.b = b; a.tr_ids = tr ? tr->ids : nullptr;
        a.nlive_ub = B;
        // the moved rows are the next block's input: write its LN1 on the way
        if (b < L) {
          a.ln_g = m->blk[b].ln1_g;
          a.ln_b = m->blk[b].ln1_b;
          a.ln_out = m->act;
        }
        HIP_OR_FAIL(launch_compact<T>(a, s));
        ln1_done = b < L;
        cur = nx;
      }
      if (isP) {
        const int keep_ub = (int)std::floor(tau_eff * (double)(T_ub - 1));
        T_ub = 1 + keep_ub;
      }
    }
  }
  *cur_out = cur;
  if (o.stop_block > 0) return FUSION_OK;
  {
    Prof p(m, s, K_FINAL_HEAD);
    HIP_OR_FAIL(launch_layernorm<T>(m->x, m->rmap[cur], m->norm_g, m->norm_b, (T*)m->hc, d, m->cnt[cur],
                                    m->cu[cur], m->live[cur], 1, B, exit_block, L, s));
    Epi e{EPI_F32, logits, c.C, m->head_b, m->live[cur], nullptr, 0};
    HIP_OR_FAIL(launch_gemm<T>((const T*)m->hc, d, (const T*)m->head_w, c.C, d,
                               &m->cnt[cur]->nlive, 0, B, e, s));
  }
  return FUSION_OK;
}

int check_model(const fusion_model* m) {
  if (!m) return fail(FUSION_E_INVALID_ARG, "model is null");
  return FUSION_OK;
}

int run_common(fusion_model* m, const float* images, int B, float* logits,
               int32_t* exit_block, int32_t* token_counts, const RunOpts& o,
               void* stream, int* cur_out) {
  if (int rc = check_model(m)) return rc;
  if (!images || !logits || !exit_block || !token_counts)
    return fail(FUSION_E_INVALID_ARG, "null buffer");
  if (B < 1) return fail(FUSION_E_INVALID_ARG, "batch must be >= 1");
  if (B > m->max_batch) return fail(FUSION_E_CAPACITY, "batch exceeds max_batch");
  HIP_OR_FAIL(hipSetDevice(m->device));
  hipStream_t s = (hipStream_t)stream;
  if (m->cfg.precision == 1)
    return run_impl<bf16_t>(m, images, B, logits, exit_block, token_counts, o, s, cur_out);
  return run_impl<float>(m, images, B, logits, exit_block, token_counts, o, s, cur_out);
}

}  // namespace

extern "C" {

FUSION_API const char* fusion_last_error(void) { return g_err.c_str(); }

FUSION_API int fusion_blob_inspect(const void* blob, size_t blob_bytes, fusion_info* out) {
  if (!out) return fail(FUSION_E_INVALID_ARG, "info is null");
  Config c;
  std::vector<TensorRef> t;
  if (int rc = parse_blob(blob, blob_bytes, c, t)) return rc;
  fill_info(c, out);
  return FUSION_OK;
}

FUSION_API int fusion_model_create(const void* blob, size_t blob_bytes, int max_batch,
                                   fusion_model** out) {
  if (!out) return fail(FUSION_E_INVALID_ARG, "out is null");
  *out = nullptr;
  if (max_batch < 1 || max_batch > 65536) return fail(FUSION_E_INVALID_ARG, "max_batch out of range");
  Config c;
  std::vector<TensorRef> tensors;
  if (int rc = parse_blob(blob, blob_bytes, c, tensors)) return rc;

  fusion_model* m = new fusion_model();
  m->cfg = c;
  m->max_batch = max_batch;
  for (size_t k = 0; k < c.exits.size(); k++) m->delta[k] = c.delta_b[c.exits[k] - 1];
  int rc = FUSION_OK;
  auto bail = [&](int code) {
    release_all(m);
    delete m;
    return code;
  };
  if (hipGetDevice(&m->device) != hipSuccess) {
    return bail(fail(FUSION_E_HIP, "no HIP device"));
  }
  // ---- weights: all fp32 tensors in one buffer, matrix weights converted
  size_t total = 0;
  std::vector<size_t> foff(tensors.size());
  for (size_t k = 0; k < tensors.size(); k++) {
    foff[k] = total;
    total += (tensors[k].nbytes + 255) / 256 * 256;
  }
  std::vector<uint8_t> host(total, 0);
  const uint8_t* bp = (const uint8_t*)blob;
  for (size_t k = 0; k < tensors.size(); k++)
    std::memcpy(host.data() + foff[k], bp + tensors[k].offset, tensors[k].nbytes);
  m->wf32 = (float*)dev_alloc<float>(m, total, &rc);
  if (!m->wf32) return bail(rc);
  if (hipMemcpy(m->wf32, host.data(), total, hipMemcpyHostToDevice) != hipSuccess)
    return bail(fail(FUSION_E_HIP, "weight upload failed"));
  auto is_matrix = [](const std::string& n) {
    const std::string leaf = n.substr(n.find('.') == std::string::npos ? 0 : n.find('.') + 1);
    return leaf == "pe_w" || leaf == "qkv_w" || leaf == "proj_w" || leaf == "fc1_w" ||
           leaf == "fc2_w" || leaf == "ew" || leaf == "ew1" || leaf == "ew2" ||
           leaf == "head_w";
  };
  std::vector<size_t> boff(tensors.size(), 0);
  if (c.precision == 1) {
    size_t btot = 0;
    for (size_t k = 0; k < tensors.size(); k++)
      if (is_matrix(tensors[k].name)) {
        boff[k] = btot;
        btot += (tensors[k].nbytes / 2 + 255) / 256 * 256;
      }
    std::vector<uint16_t> hb(btot / 2, 0);
    for (size_t k = 0; k < tensors.size(); k++)
      if (is_matrix(tensors[k].name)) {
        const float* src = (const float*)(host.data() + foff[k]);
        const size_t n = tensors[k].nbytes / 4;
        for (size_t q = 0; q < n; q++) hb[boff[k] / 2 + q] = host_bf16(src[q]);
      }
    m->wmat = dev_alloc<uint16_t>(m, btot, &rc);
    if (!m->wmat) return bail(rc);
    if (hipMemcpy(m->wmat, hb.data(), btot, hipMemcpyHostToDevice) != hipSuccess)
      return bail(fail(FUSION_E_HIP, "weight upload failed"));
  }
  auto F = [&](const std::string& n) -> const float* {
    for (size_t k = 0; k < tensors.size(); k++)
      if (tensors[k].name == n) return (const float*)((uint8_t*)m->wf32 + foff[k]);
    return nullptr;
  };
  auto Wm = [&](const std::string& n) -> const void* {
    for (size_t k = 0; k < tensors.size(); k++)
      if (tensors[k].name == n)
        return c.precision == 1 ? (const void*)((uint8_t*)m->wmat + boff[k])
                                : (const void*)((uint8_t*)m->wf32 + foff[k]);
    return nullptr;
  };
  m->cls = F("cls"); m->pos = F("pos"); m->pe_b = F("pe_b"); m->pe_w = Wm("pe_w");
  m->norm_g = F("norm_g"); m->norm_b = F("norm_b"); m->head_b = F("head_b");
  m->head_w = Wm("head_w");
  for (int b = 1; b <= c.L; b++) {
    const std::string p = "blk" + std::to_string(b) + ".";
    BlockW& w = m->blk[b - 1];
    w.ln1_g = F(p + "ln1_g"); w.ln1_b = F(p + "ln1_b"); w.qkv_b = F(p + "qkv_b");
    w.proj_b = F(p + "proj_b"); w.ln2_g = F(p + "ln2_g"); w.ln2_b = F(p + "ln2_b");
    w.fc1_b = F(p + "fc1_b"); w.fc2_b = F(p + "fc2_b");
    w.qkv_w = Wm(p + "qkv_w"); w.proj_w = Wm(p + "proj_w"); w.fc1_w = Wm(p + "fc1_w");
    w.fc2_w = Wm(p + "fc2_w");
    w.router_w = F(p + "router_w"); w.router_b = F(p + "router_b");
    w.eln_g = F(p + "eln_g"); w.eln_b = F(p + "eln_b"); w.eb = F(p + "eb"); w.ew = Wm(p + "ew");
    w.eb1 = F(p + "eb1"); w.eb2 = F(p + "eb2"); w.ew1 = Wm(p + "ew1"); w.ew2 = Wm(p + "ew2");
    w.prune_w = F(p + "prune_w"); w.prune_b = F(p + "prune_b");
  }
  // ---- workspace
  const size_t esz = c.precision == 1 ? 2 : 4;
  const size_t Mmax = (size_t)max_batch * (c.n0 + 1);
  const size_t ffn_cols = std::max<size_t>(c.mlp, c.pdim);
  // x offsets are 32-bit in the adapt kernel's similarity loads
  if (Mmax * (size_t)c.d > (size_t)INT32_MAX)
    return bail(fail(FUSION_E_CAPACITY,
                     "max_batch too large: the residual stream would exceed 2^31 elements"));
  // the GEMM loads address their operands with 32-bit byte offsets
  if (Mmax * std::max<size_t>(ffn_cols, 3 * (size_t)c.d) * esz > 0xFFFFFFFFull)
    return bail(fail(FUSION_E_CAPACITY,
                     "max_batch too large: a GEMM operand would exceed 4 GiB"));
  m->x = (float*)dev_alloc<float>(m, Mmax * c.d * 4, &rc);
  for (int k = 0; k < 2; k++) {
    m->rmap[k] = (int*)dev_alloc<int>(m, Mmax * 4, &rc);
    m->size[k] = (float*)dev_alloc<float>(m, Mmax * 4, &rc);
    m->origin[k] = (int*)dev_alloc<int>(m, Mmax * 4, &rc);
    m->cu[k] = (int*)dev_alloc<int>(m, (max_batch + 1) * 4, &rc);
    m->live[k] = (int*)dev_alloc<int>(m, max_batch * 4, &rc);
    m->cnt[k] = (LiveCounts*)dev_alloc<int>(m, sizeof(LiveCounts), &rc);
    if (rc) return bail(rc);
  }
  m->act = dev_alloc<char>(m, Mmax * c.d * esz, &rc);
  m->qkv = dev_alloc<char>(m, Mmax * 3 * c.d * esz, &rc);
  m->ffn = dev_alloc<char>(m, Mmax * ffn_cols * esz, &rc);
  m->hc = dev_alloc<char>(m, (size_t)max_batch * c.d * esz, &rc);
  m->hbuf = dev_alloc<char>(m, (size_t)max_batch * std::max(c.exit_hidden, 1) * esz, &rc);
  m->head_buf = (float*)dev_alloc<float>(m, (size_t)max_batch * c.C * 4, &rc);
  m->cls_scores = (float*)dev_alloc<float>(m, (size_t)max_batch * c.heads * (c.n0 + 1) * 4, &rc);
  m->keep = (int*)dev_alloc<int>(m, Mmax * 4, &rc);
  m->newlen = (int*)dev_alloc<int>(m, (size_t)max_batch * 4, &rc);
  m->sim_v = (float*)dev_alloc<float>(m, (size_t)max_batch * AD_SIM_STRIDE * 4, &rc);
  m->sim_i = (int*)dev_alloc<int>(m, (size_t)max_batch * AD_SIM_STRIDE * 4, &rc);
  if (rc) return bail(rc);
  *out = m;
  return FUSION_OK;
}

FUSION_API int fusion_model_destroy(fusion_model* m) {
  if (!m) return fail(FUSION_E_INVALID_ARG, "model is null");
  hipSetDevice(m->device);
  hipDeviceSynchronize();
  release_all(m);
  delete m;
  return FUSION_OK;
}

FUSION_API int fusion_model_info(const fusion_model* m, fusion_info* out) {
  if (!m || !out) return fail(FUSION_E_INVALID_ARG, "null argument");
  fill_info(m->cfg, out);
  out->max_batch = m->max_batch;
  for (size_t k = 0; k < m->cfg.exits.size(); k++) out->delta[k] = m->delta[k];
  out->rho = m->rho;
  return FUSION_OK;
}

FUSION_API int fusion_set_exit_thresholds(fusion_model* m, const float* delta, int n_exit) {
  if (!m || !delta) return fail(FUSION_E_INVALID_ARG, "null argument");
  if (n_exit != (int)m->cfg.exits.size()) return fail(FUSION_E_INVALID_ARG, "n_exit != number of exit heads");
  for (int k = 0; k < n_exit; k++)
    if (!(delta[k] >= 0.f && delta[k] <= 1.f)) return fail(FUSION_E_INVALID_ARG, "threshold outside [0, 1]");
  for (int k = 0; k < n_exit; k++) m->delta[k] = delta[k];
  return FUSION_OK;
}

FUSION_API int fusion_set_router_strength(fusion_model* m, double rho) {
  if (!m) return fail(FUSION_E_INVALID_ARG, "model is null");
  if (!(rho >= 0.0 && rho <= 16.0)) return fail(FUSION_E_INVALID_ARG, "rho outside [0, 16]");
  m->rho = rho;
  return FUSION_OK;
}

FUSION_API int fusion_run(fusion_model* m, const float* images, int batch, float* logits,
                          int32_t* exit_block, int32_t* token_counts, void* stream) {
  RunOpts o;
  int cur = 0;
  return run_common(m, images, batch, logits, exit_block, token_counts, o, stream, &cur);
}

FUSION_API int fusion_run_traced(fusion_model* m, const float* images, int batch,
                                 float* logits, int32_t* exit_block, int32_t* token_counts,
                                 const fusion_trace* trace, void* stream) {
  if (!trace) return fail(FUSION_E_INVALID_ARG, "trace is null");
  RunOpts o;
  o.trace = trace;
  int cur = 0;
  return run_common(m, images, batch, logits, exit_block, token_counts, o, stream, &cur);
}

FUSION_API int fusion_debug_state(fusion_model* m, const float* images, int batch, int block,
                                  int stage, float* x_out, int32_t* cu_out, int32_t* live_out,
                                  int* n_live, void* stream) {
  if (int rc = check_model(m)) return rc;
  if (!x_out || !cu_out || !live_out || !n_live) return fail(FUSION_E_INVALID_ARG, "null buffer");
  if (stage < 0 || stage > 2) return fail(FUSION_E_INVALID_ARG, "stage must be 0, 1 or 2");
  if (stage > 0 && (block < 1 || block > m->cfg.L)) return fail(FUSION_E_INVALID_ARG, "bad block");
  if (batch < 1) return fail(FUSION_E_INVALID_ARG, "batch must be >= 1");
  if (batch > m->max_batch) return fail(FUSION_E_CAPACITY, "batch exceeds max_batch");
  HIP_OR_FAIL(hipSetDevice(m->device));
  hipStream_t s = (hipStream_t)stream;
  // scratch outputs for the run itself
  float* lg = nullptr;
  int32_t *eb = nullptr, *tc = nullptr;
  HIP_OR_FAIL(hipMalloc(&lg, (size_t)batch * m->cfg.C * 4));
  HIP_OR_FAIL(hipMalloc(&eb, (size_t)batch * 4));
  HIP_OR_FAIL(hipMalloc(&tc, (size_t)batch * m->cfg.L * 4));
  RunOpts o;
  o.stop_block = stage == 0 ? 1 : block;
  o.stop_stage = stage;
  int cur = 0;
  int rc = run_common(m, images, batch, lg, eb, tc, o, stream, &cur);
  if (rc == FUSION_OK) {
    hipError_t e = launch_copy_state(m->x, m->rmap[cur], m->cu[cur], m->live[cur], m->cnt[cur], x_out,
                                     cu_out, live_out, m->cfg.d, batch * (m->cfg.n0 + 1), batch, s);
    LiveCounts hc{};
    if (e == hipSuccess) e = hipMemcpyAsync(&hc, m->cnt[cur], sizeof(hc), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) rc = fail(FUSION_E_HIP, hipGetErrorString(e));
    *n_live = hc.nlive;
  }
  hipStreamSynchronize(s);
  hipFree(lg);
  hipFree(eb);
  hipFree(tc);
  return rc;
}

FUSION_API int fusion_debug_poison_workspace(fusion_model* m, void* stream) {
  if (int rc = check_model(m)) return rc;
  HIP_OR_FAIL(hipSetDevice(m->device));
  hipStream_t s = (hipStream_t)stream;
  const Config& c = m->cfg;
  const size_t esz = c.precision == 1 ? 2 : 4;
  const size_t Mmax = (size_t)m->max_batch * (c.n0 + 1);
  const size_t ffn_cols = std::max<size_t>(c.mlp, c.pdim);
  // all-ones bytes: NaN in fp32 and in bf16
  struct Buf { void* p; size_t bytes; };
  const Buf bufs[] = {
      {m->x, Mmax * c.d * 4},
      {m->size[0], Mmax * 4}, {m->size[1], Mmax * 4},
      {m->act, Mmax * c.d * esz},
      {m->qkv, Mmax * 3 * c.d * esz},
      {m->ffn, Mmax * ffn_cols * esz},
      {m->hc, (size_t)m->max_batch * c.d * esz},
      {m->hbuf, (size_t)m->max_batch * std::max(c.exit_hidden, 1) * esz},
      {m->head_buf, (size_t)m->max_batch * c.C * 4},
      {m->cls_scores, (size_t)m->max_batch * c.heads * (c.n0 + 1) * 4},
      {m->sim_v, (size_t)m->max_batch * AD_SIM_STRIDE * 4},
  };
  for (const Buf& b : bufs) HIP_OR_FAIL(hipMemsetAsync(b.p, 0xFF, b.bytes, s));
  return FUSION_OK;
}

FUSION_API int fusion_profile_enable(fusion_model* m, int on) {
  if (!m) return fail(FUSION_E_INVALID_ARG, "model is null");
  for (auto& r : m->recs) {
    hipEventSynchronize(r.b);
    m->pool.push_back(r.a);
    m->pool.push_back(r.b);
  }
  m->recs.clear();
  m->prof = on != 0;
  for (int k = 0; k < K_COUNT; k++) {
    m->tot_ms[k] = 0;
    m->launches[k] = 0;
  }
  return FUSION_OK;
}

FUSION_API int fusion_profile_kinds(void) { return K_COUNT; }

FUSION_API const char* fusion_profile_kind_name(int k) {
  if (k < 0 || k >= K_COUNT) return "";
  return kKindNames[k];
}

FUSION_API int fusion_profile_read(fusion_model* m, int k, double* total_ms, int64_t* launches) {
  if (!m || !total_ms || !launches) return fail(FUSION_E_INVALID_ARG, "null argument");
  if (k < 0 || k >= K_COUNT) return fail(FUSION_E_INVALID_ARG, "bad kind");
  for (auto& r : m->recs) {
    if (hipEventSynchronize(r.b) != hipSuccess) return fail(FUSION_E_HIP, "event sync failed");
    float ms = 0.f;
    hipEventElapsedTime(&ms, r.a, r.b);
    m->tot_ms[r.kind] += ms;
    m->launches[r.kind] += 1;
    m->pool.push_back(r.a);
    m->pool.push_back(r.b);
  }
  m->recs.clear();
  *total_ms = m->tot_ms[k];
  *launches = m->launches[k];
  return FUSION_OK;
}

}  // extern "C"
