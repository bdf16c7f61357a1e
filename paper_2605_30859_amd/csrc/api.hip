// C ABI of the rollout library: context, memory plan, per-step launch
// sequence, selection/pruning, statistics, and the stateless kernel entries.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <new>
#include <string>
#include <vector>

#include "../../include/darts.h"
#include "common.h"
#include "kernels.h"

using namespace darts;

enum : uint32_t { T_EMBED = 0, T_WQ, T_WK, T_WV, T_WO, T_WGATE, T_WUP, T_WDOWN, T_LM,
                  T_ROUTER, T_EGATE, T_EUP, T_EDOWN };

namespace {

struct LayerW {
  void* wqkv = nullptr;   // [(hq + 2 hkv) hd][d]
  void* wo = nullptr;     // [d][hq hd]
  void* wgu = nullptr;    // [2F][d], gate/up interleaved in groups of 16 rows (dense)
  void* wdown = nullptr;  // [d][F] (dense)
  void* wrouter = nullptr;  // [E][d] (MoE)
  void* wegu = nullptr;     // [E][2Fe][d], per expert gate/up interleaved in groups of 16
  void* wedown = nullptr;   // [E][d][Fe]
};

struct TimedLaunch {
  int kind;        // 0 attention (decode), 1.. GEMM class + 1 (QKV, O, gate-up, down, LM head)
  double units;    // algorithmic bytes (attention) or FLOP (GEMM)
  double weight;   // launches of the whole run this one stands for
  double units_grp = 0.0;   // attention with a shared prefix: bytes per live prompt group
  double traj_units = 0.0;  // attention: bytes if every row read its whole context itself
  int touched_slot = -1;    // grouped expert GEMMs: slot of the launch's touched-expert count
  double rows = 0.0;        // grouped expert GEMMs: routed (row, expert) pairs
};

// With timing on, events are recorded in the prefill and in every
// kTimingStride-th decode step only (an event pair per launch costs about a
// tenth of the decode time); each timed decode launch stands for kTimingStride.
constexpr int kTimingStride = 8;

}  // namespace

struct darts_ctx {
  darts_model_cfg mc{};
  darts_run_cfg rc{};
  int m = 0, k = 0, L = 1, m_up = 0;
  hipStream_t st = nullptr;
  bool bf16 = false;
  size_t esz = 4;
  int P = 0, Lp = 0, cap = 0, pp = 0, max_pages = 0, n_traj = 0;
  int64_t n_pages = 0;
  int d = 0, hq = 0, hkv = 0, hd = 0, F = 0, V = 0, nl = 0, qkv_w = 0;
  bool moe = false;
  int E = 0, topk = 0, Fe = 0, Epad = 0;   // Epad: router rows padded to a multiple of 128
  int32_t* m_topk_id = nullptr;
  float* m_topk_w = nullptr;
  int32_t* m_pos_of = nullptr;
  int32_t* m_cnt = nullptr;       // counts | offsets | cursors, E each
  int32_t* m_row_of = nullptr;    // [pairs] input row of each expert-sorted position
  void* m_h_perm = nullptr;
  void* m_y_perm = nullptr;
  float* m_logits = nullptr;      // router logits [rows][Epad]
  int32_t* m_mtiles = nullptr;    // n_mtiles | non-empty expert row tiles (gate/up)
  int32_t* m_mtiles_dn = nullptr; // the same for the down projection
  int32_t* m_touched = nullptr;   // [n_layers] experts that received rows (timed launches)
  int32_t* h_touched = nullptr;   // pinned host copy
  // routing verification (darts_debug_moe_routing)
  const int32_t* dbg_force_ids = nullptr;
  int32_t* dbg_own_ids = nullptr;
  float* dbg_used_p = nullptr;
  // device memory
  std::vector<void*> allocs;
  void* embed = nullptr;
  void* lm_head = nullptr;
  std::vector<LayerW> layers;
  void* kpool = nullptr;
  void* vpool = nullptr;
  int64_t pool_layer_elems = 0;
  float2* rope = nullptr;
  int32_t* page_table = nullptr;
  int32_t* free_stack = nullptr;
  int32_t* dcnt = nullptr;        // [0] free_top, [4..7] info
  int32_t* gen = nullptr;
  float* sum_lp = nullptr;
  uint8_t* status = nullptr;
  uint8_t* freed = nullptr;
  int32_t* last_tok = nullptr;
  int32_t* forced_len = nullptr;
  int32_t* refcnt = nullptr;
  uint8_t* group_done = nullptr;
  int32_t* done_step = nullptr;
  int32_t* kept = nullptr;
  int32_t* live[2] = {nullptr, nullptr};
  int32_t* grp_m = nullptr;        // [P] candidates per prompt (redundancy plan M'_i)
  // token-chunk streaming (DARTS_FLAG_STREAM): per-trajectory token/log-prob
  // history [n_traj][cap], tokens already dispatched, final marks sent
  int32_t* hist_tok = nullptr;
  float* hist_lp = nullptr;
  int32_t* streamed = nullptr;
  uint8_t* fin_sent = nullptr;
  int32_t* stream_off = nullptr;
  // sampler slice partials (rows split across blocks when few are live)
  SamplePart* samp_parts = nullptr;
  int64_t samp_part_cap = 0;
  std::vector<int32_t> plan;       // host copy of grp_m
  int n_start = 0;                 // sum of the plan: trajectories started by the prefill
  int32_t* grp_cnt = nullptr;
  int32_t* grp_rel = nullptr;
  int32_t* trj_cnt = nullptr;
  int32_t* prefill_pt = nullptr;   // [P*Lp] page-table row of each prompt position
  int32_t* last_rows = nullptr;    // [P] index of each prompt's last position
  float* x = nullptr;
  void* xn = nullptr;
  float* qkv = nullptr;
  void* q = nullptr;
  void* attn = nullptr;
  void* hbuf = nullptr;
  float* xlast = nullptr;
  float* logits = nullptr;
  void* gemm_ws = nullptr;
  size_t gemm_ws_bytes = 0;
  void* attn_ws = nullptr;
  size_t attn_ws_bytes = 0;
  bool share_prefix = false;      // decode attention reads each prompt's pages once per group
  int32_t* h_info = nullptr;       // pinned host
  // host state
  int phase = 0;                   // 0 init, 1 decoding, 2 done
  int cur = 0;
  int n_live = 0;
  int n_done = 0;
  int free_top = 0;
  int64_t step = 0;
  int64_t tokens = 0;
  int64_t hwm = 0;
  int last_rows_out = 0;
  bool poisoned = false;
  double timed_weight = 0.0;       // > 0 while the current step's launches are timed
  std::string err;
  std::vector<TimedLaunch> pending;
  std::vector<hipEvent_t> events;  // pool, two per pending launch
  // per-step wall time on the device (DARTS_FLAG_STEP_TIMES): from the start
  // of a sampling step's first launch to the end of its selection kernel
  hipEvent_t step_ev[2] = {nullptr, nullptr};
  int step_rows = 0;               // rows of the open step, -1 for the prefill, 0 none
  std::vector<int32_t> st_rows;
  std::vector<float> st_ms;
  float prefill_ms = 0.f;
  double attn_ms = 0.0, attn_bytes = 0.0, attn_traj_bytes = 0.0;
  int64_t attn_launches = 0;
  double gemm_ms = 0.0, gemm_flop = 0.0;
  int64_t gemm_launches = 0;
  double cls_ms[6] = {0, 0, 0, 0, 0, 0}, cls_flop[6] = {0, 0, 0, 0, 0, 0};
  double moe_ms[2] = {0, 0}, moe_bytes[2] = {0, 0};
  int64_t moe_launches[2] = {0, 0};
};

#define HIPCHK(ctx, expr)                                                      \
  do {                                                                         \
    hipError_t _e = (expr);                                                    \
    if (_e != hipSuccess) return fail_hip((ctx), _e, #expr);                   \
  } while (0)

static int fail_hip(darts_ctx* c, hipError_t e, const char* what) {
  if (c) {
    c->poisoned = true;
    c->err = std::string(what) + ": " + hipGetErrorString(e);
  }
  return DARTS_EHIP;
}

template <typename T>
static hipError_t dalloc(darts_ctx* c, T** p, size_t bytes) {
  void* v = nullptr;
  hipError_t e = hipMalloc(&v, bytes ? bytes : 256);
  if (e == hipSuccess) {
    c->allocs.push_back(v);
    *p = (T*)v;
  }
  return e;
}

static void free_all(darts_ctx* c) {
  for (void* p : c->allocs) (void)hipFree(p);
  c->allocs.clear();
  if (c->h_info) (void)hipHostFree(c->h_info);
  c->h_info = nullptr;
  if (c->h_touched) (void)hipHostFree(c->h_touched);
  c->h_touched = nullptr;
  for (hipEvent_t e : c->events) (void)hipEventDestroy(e);
  c->events.clear();
  c->pending.clear();
  for (hipEvent_t& e : c->step_ev) {
    if (e) (void)hipEventDestroy(e);
    e = nullptr;
  }
}

static bool step_times_on(const darts_ctx* c) { return (c->rc.flags & DARTS_FLAG_STEP_TIMES) != 0; }

// Open the timed interval of a sampling step (rows -1: the prefill).
static hipError_t step_begin(darts_ctx* c, int rows) {
  if (!step_times_on(c)) return hipSuccess;
  c->step_rows = rows;
  return hipEventRecord(c->step_ev[0], c->st);
}

static bool timing_on(const darts_ctx* c) { return (c->rc.flags & DARTS_FLAG_TIMING) != 0; }

// Record the start event of a timed launch; returns its index or -1.
static int tbegin(darts_ctx* c, int kind, double units) {
  if (c->timed_weight <= 0.0) return -1;
  const size_t i = c->pending.size();
  while (c->events.size() < 2 * (i + 1)) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return -1;
    c->events.push_back(e);
  }
  if (hipEventRecord(c->events[2 * i], c->st) != hipSuccess) return -1;
  c->pending.push_back(TimedLaunch{kind, units, c->timed_weight});
  return (int)i;
}
// Reserve an event pair without recording (the launcher records it).
static int treserve(darts_ctx* c, int kind, double units) {
  if (c->timed_weight <= 0.0) return -1;
  const size_t i = c->pending.size();
  while (c->events.size() < 2 * (i + 1)) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return -1;
    c->events.push_back(e);
  }
  c->pending.push_back(TimedLaunch{kind, units, c->timed_weight});
  return (int)i;
}
static void tend(darts_ctx* c, int i) {
  if (i >= 0) (void)hipEventRecord(c->events[2 * i + 1], c->st);
}

static int init_weights(darts_ctx* c) {
  const int d = c->d, hq = c->hq, hkv = c->hkv, hd = c->hd, F = c->F, V = c->V;
  const bool b = c->bf16;
  const uint64_t seed = c->mc.weight_seed;
  HIPCHK(c, launch_init_weights(c->embed, b, V, d, 1, T_EMBED, 0, seed, rowmap_plain(V, 0), c->st));
  HIPCHK(c, launch_init_weights(c->lm_head, b, V, d, d, T_LM, 0, seed, rowmap_plain(V, 0), c->st));
  for (int l = 0; l < c->nl; ++l) {
    LayerW& w = c->layers[l];
    HIPCHK(c, launch_init_weights(w.wqkv, b, (int64_t)hq * hd, d, d, T_WQ, l, seed,
                                  rowmap_plain(hq * hd, 0), c->st));
    HIPCHK(c, launch_init_weights(w.wqkv, b, (int64_t)hkv * hd, d, d, T_WK, l, seed,
                                  rowmap_plain(hkv * hd, hq * hd), c->st));
    HIPCHK(c, launch_init_weights(w.wqkv, b, (int64_t)hkv * hd, d, d, T_WV, l, seed,
                                  rowmap_plain(hkv * hd, (hq + hkv) * hd), c->st));
    HIPCHK(c, launch_init_weights(w.wo, b, d, (int64_t)hq * hd, (int64_t)hq * hd, T_WO, l, seed,
                                  rowmap_plain(d, 0), c->st));
    if (c->moe) {
      const int E = c->E, Fe = c->Fe;
      HIPCHK(c, launch_init_weights(w.wrouter, b, E, d, d, T_ROUTER, l, seed, rowmap_plain(E, 0), c->st));
      if (c->Epad > E)   // padding rows of the router: zero logits, never selected
        HIPCHK(c, hipMemsetAsync((char*)w.wrouter + (size_t)E * d * c->esz, 0,
                                 (size_t)(c->Epad - E) * d * c->esz, c->st));
      RowMap eg{Fe, 2 * (int64_t)Fe, 16, 32, 0}, eu{Fe, 2 * (int64_t)Fe, 16, 32, 16};
      HIPCHK(c, launch_init_weights(w.wegu, b, (int64_t)E * Fe, d, d, T_EGATE, l, seed, eg, c->st));
      HIPCHK(c, launch_init_weights(w.wegu, b, (int64_t)E * Fe, d, d, T_EUP, l, seed, eu, c->st));
      HIPCHK(c, launch_init_weights(w.wedown, b, (int64_t)E * d, Fe, Fe, T_EDOWN, l, seed,
                                    rowmap_plain((int64_t)E * d, 0), c->st));
      continue;
    }
    RowMap gate{F, 0, 16, 32, 0}, up{F, 0, 16, 32, 16};
    HIPCHK(c, launch_init_weights(w.wgu, b, F, d, d, T_WGATE, l, seed, gate, c->st));
    HIPCHK(c, launch_init_weights(w.wgu, b, F, d, d, T_WUP, l, seed, up, c->st));
    HIPCHK(c, launch_init_weights(w.wdown, b, d, F, F, T_WDOWN, l, seed, rowmap_plain(d, 0), c->st));
  }
  return DARTS_OK;
}

// The caller's tensors (model->weights, in the order darts_weight_count
// documents) copied into the same physical layout init_weights generates.
static int copy_weights(darts_ctx* c) {
  const int d = c->d, hq = c->hq, hkv = c->hkv, hd = c->hd, F = c->F, V = c->V;
  const bool b = c->bf16;
  const void* const* src = c->mc.weights;
  int t = 0;
  HIPCHK(c, launch_copy_rows(c->embed, src[t++], b, V, d, rowmap_plain(V, 0), c->st));
  HIPCHK(c, launch_copy_rows(c->lm_head, src[t++], b, V, d, rowmap_plain(V, 0), c->st));
  for (int l = 0; l < c->nl; ++l) {
    LayerW& w = c->layers[l];
    HIPCHK(c, launch_copy_rows(w.wqkv, src[t++], b, (int64_t)hq * hd, d, rowmap_plain(hq * hd, 0), c->st));
    HIPCHK(c, launch_copy_rows(w.wqkv, src[t++], b, (int64_t)hkv * hd, d, rowmap_plain(hkv * hd, hq * hd),
                               c->st));
    HIPCHK(c, launch_copy_rows(w.wqkv, src[t++], b, (int64_t)hkv * hd, d,
                               rowmap_plain(hkv * hd, (hq + hkv) * hd), c->st));
    HIPCHK(c, launch_copy_rows(w.wo, src[t++], b, d, (int64_t)hq * hd, rowmap_plain(d, 0), c->st));
    if (c->moe) {
      const int E = c->E, Fe = c->Fe;
      HIPCHK(c, launch_copy_rows(w.wrouter, src[t++], b, E, d, rowmap_plain(E, 0), c->st));
      if (c->Epad > E)   // padding rows of the router: zero logits, never selected
        HIPCHK(c, hipMemsetAsync((char*)w.wrouter + (size_t)E * d * c->esz, 0,
                                 (size_t)(c->Epad - E) * d * c->esz, c->st));
      RowMap eg{Fe, 2 * (int64_t)Fe, 16, 32, 0}, eu{Fe, 2 * (int64_t)Fe, 16, 32, 16};
      HIPCHK(c, launch_copy_rows(w.wegu, src[t++], b, (int64_t)E * Fe, d, eg, c->st));
      HIPCHK(c, launch_copy_rows(w.wegu, src[t++], b, (int64_t)E * Fe, d, eu, c->st));
      HIPCHK(c, launch_copy_rows(w.wedown, src[t++], b, (int64_t)E * d, Fe, rowmap_plain((int64_t)E * d, 0),
                                 c->st));
      continue;
    }
    RowMap gate{F, 0, 16, 32, 0}, up{F, 0, 16, 32, 16};
    HIPCHK(c, launch_copy_rows(w.wgu, src[t++], b, F, d, gate, c->st));
    HIPCHK(c, launch_copy_rows(w.wgu, src[t++], b, F, d, up, c->st));
    HIPCHK(c, launch_copy_rows(w.wdown, src[t++], b, d, F, rowmap_plain(d, 0), c->st));
  }
  // the copies are complete before darts_init returns (it synchronises the
  // stream), after which the context keeps no reference to the caller's array
  return DARTS_OK;
}

// The experts' gate/up matrices ([E][2Fe][d], generated or copied row-major)
// are reordered in place into the strip layout their grouped GEMM reads.
static int pack_expert_weights(darts_ctx* c) {
  for (int l = 0; l < c->nl; ++l)
    HIPCHK(c, launch_pack_strips(c->layers[l].wegu, (int64_t)c->E * 2 * c->Fe, c->d, c->st));
  return DARTS_OK;
}

static size_t gemm_ws_need(const darts_ctx* c) {
  // every row count a launch can see: decode batches 1..n_traj, the prefill
  // (P*Lp rows) and the prefill's LM head (P rows)
  size_t need = 0;
  std::vector<int> ms;
  for (int M = 1; M <= c->n_traj; ++M) ms.push_back(M);
  ms.push_back(c->P);
  ms.push_back(c->P * c->Lp);
  for (int M : ms) {
    need = std::max(need, gemm_workspace_bytes(M, c->qkv_w, c->d));
    need = std::max(need, gemm_workspace_bytes(M, c->d, c->hq * c->hd));
    if (!c->moe) {
      need = std::max(need, gemm_workspace_bytes(M, 2 * c->F, c->d));
      need = std::max(need, gemm_workspace_bytes(M, c->d, c->F));
    } else {
      need = std::max(need, gemm_workspace_bytes(M, c->Epad, c->d));   // router
    }
    need = std::max(need, gemm_workspace_bytes(M, c->V, c->d));
  }
  return need;
}

extern "C" {

const char* darts_strerror(int s) {
  switch (s) {
    case DARTS_OK: return "ok";
    case DARTS_EINVAL: return "invalid argument";
    case DARTS_ENOMEM: return "out of memory (device memory or KV page pool)";
    case DARTS_ESTATE: return "call out of order";
    case DARTS_EHIP: return "HIP runtime error";
  }
  return "unknown status";
}

const char* darts_last_error(const darts_ctx* c) { return c ? c->err.c_str() : ""; }

// Upload the redundancy plan: per-prompt candidate counts, the initial live
// list (existing candidates g = i*m + j, j < M'_i, ascending) and statuses
// (absent candidates j >= M'_i never run).  Synchronises the stream.
static hipError_t upload_plan(darts_ctx* c) {
  std::vector<int32_t> live;
  std::vector<uint8_t> st((size_t)c->n_traj, 4);
  live.reserve(c->n_traj);
  for (int i = 0; i < c->P; ++i)
    for (int j = 0; j < c->plan[i]; ++j) {
      live.push_back(i * c->m + j);
      st[(size_t)i * c->m + j] = 0;
    }
  c->n_start = (int)live.size();
  hipError_t e = hipMemcpyAsync(c->grp_m, c->plan.data(), (size_t)c->P * 4, hipMemcpyHostToDevice, c->st);
  if (e == hipSuccess)
    e = hipMemcpyAsync(c->live[0], live.data(), live.size() * 4, hipMemcpyHostToDevice, c->st);
  if (e == hipSuccess) e = hipMemcpyAsync(c->status, st.data(), st.size(), hipMemcpyHostToDevice, c->st);
  if (e == hipSuccess) e = hipStreamSynchronize(c->st);
  return e;
}

// Bytes of caller weight tensor i (the order of darts_model_cfg.weights).
static int64_t caller_weight_bytes(const darts_model_cfg& mc, int32_t i) {
  const int64_t d = mc.d_model, V = mc.vocab, qd = (int64_t)mc.n_q_heads * mc.head_dim,
                kvd = (int64_t)mc.n_kv_heads * mc.head_dim, F = mc.ffn_dim, E = mc.n_experts,
                Fe = mc.expert_ffn;
  const int64_t esz = mc.dtype == DARTS_BF16 ? 2 : 4;
  if (i < 2) return V * d * esz;                        // embed, lm_head
  const int per = mc.n_experts > 0 ? 8 : 7, j = (i - 2) % per;
  int64_t n;
  if (j == 0) n = qd * d;                               // wq
  else if (j <= 2) n = kvd * d;                         // wk, wv
  else if (j == 3) n = d * qd;                          // wo
  else if (mc.n_experts > 0) n = j == 4 ? E * d : E * Fe * d;   // router; expert gate, up, down
  else n = F * d;                                       // w_gate, w_up, w_down
  return n * esz;
}

int32_t darts_weight_count(const darts_model_cfg* model) {
  if (!model || model->n_layers < 1) return 0;
  return 2 + model->n_layers * (model->n_experts > 0 ? 8 : 7);
}

int darts_init(const darts_model_cfg* model, int32_t m, int32_t k, const darts_run_cfg* run,
               darts_ctx** out) {
  if (!model || !run || !out) return DARTS_EINVAL;
  const darts_model_cfg& mc = *model;
  const darts_run_cfg& rc = *run;
  const int L = rc.L > 0 ? rc.L : 1;
  const int m_up = rc.m_up > 0 ? rc.m_up : 2 * k;
  if (k < 1 || k > m || m > 64 || L >= k) return DARTS_EINVAL;
  if (rc.page_size != 16 || rc.prompt_len < 16 || rc.prompt_len % 16 != 0) return DARTS_EINVAL;
  if (rc.n_prompts < 1 || rc.cap < 1 || rc.cap >= (1 << 20) || !(rc.temperature > 0.f))
    return DARTS_EINVAL;
  if (rc.traj_base < 0 || (int64_t)rc.traj_base + (int64_t)rc.n_prompts * m > ((int64_t)1 << 31))
    return DARTS_EINVAL;
  if (mc.n_layers < 1 || mc.d_model < 1 || mc.n_q_heads < 1 || mc.n_kv_heads < 1 ||
      mc.n_q_heads % mc.n_kv_heads != 0 || mc.n_q_heads / mc.n_kv_heads > 16)
    return DARTS_EINVAL;
  if (!(mc.head_dim == 32 || mc.head_dim == 64 || mc.head_dim == 128)) return DARTS_EINVAL;
  if (mc.vocab < 8 || mc.vocab % 4 != 0) return DARTS_EINVAL;
  if (mc.dtype != DARTS_F32 && mc.dtype != DARTS_BF16) return DARTS_EINVAL;
  const bool moe = mc.n_experts > 0;
  if (moe) {
    // grouped expert GEMMs: K/8 a multiple of 32 for both d and expert_ffn; bf16 only
    if (mc.dtype != DARTS_BF16 || mc.n_experts > 1024 || mc.top_k < 1 || mc.top_k > 64 ||
        mc.top_k > mc.n_experts || mc.expert_ffn < 256 || mc.expert_ffn % 256 != 0 ||
        mc.d_model % 256 != 0 || mc.d_model > 5120)   // 5120: a packed weight strip fits LDS
      return DARTS_EINVAL;
  } else if (mc.ffn_dim < 16 || mc.ffn_dim % 16 != 0) {
    return DARTS_EINVAL;
  }
  const int qkv_w = (mc.n_q_heads + 2 * mc.n_kv_heads) * mc.head_dim;
  if (mc.dtype == DARTS_BF16) {
    const int K1 = mc.d_model, K2 = mc.n_q_heads * mc.head_dim, K3 = mc.ffn_dim;
    if (K1 % 256 || K2 % 256 || (!moe && K3 % 256)) return DARTS_EINVAL;
    if (qkv_w % 128 || mc.d_model % 128 || (!moe && (2 * mc.ffn_dim) % 128) || mc.vocab % 128)
      return DARTS_EINVAL;
  }
  const int64_t n_traj64 = (int64_t)rc.n_prompts * m;
  if (n_traj64 > 65536 || (int64_t)rc.n_prompts * rc.prompt_len > (1 << 22)) return DARTS_EINVAL;
  if (mc.weights) {
    const int32_t nw = darts_weight_count(&mc);
    for (int32_t i = 0; i < nw; ++i)
      if (!mc.weights[i]) return DARTS_EINVAL;
  }

  darts_ctx* c = new (std::nothrow) darts_ctx();
  if (!c) return DARTS_ENOMEM;
  c->mc = mc; c->rc = rc; c->m = m; c->k = k; c->L = L; c->m_up = m_up;
  c->st = (hipStream_t)rc.stream;
  c->bf16 = mc.dtype == DARTS_BF16;
  c->esz = c->bf16 ? 2 : 4;
  c->P = rc.n_prompts; c->Lp = rc.prompt_len; c->cap = rc.cap;
  c->pp = c->Lp / kPage;
  c->max_pages = c->pp + (c->cap + kPage - 1) / kPage;
  c->n_traj = (int)n_traj64;
  c->d = mc.d_model; c->hq = mc.n_q_heads; c->hkv = mc.n_kv_heads; c->hd = mc.head_dim;
  c->F = moe ? 0 : mc.ffn_dim; c->V = mc.vocab; c->nl = mc.n_layers; c->qkv_w = qkv_w;
  c->moe = moe; c->E = mc.n_experts; c->topk = mc.top_k; c->Fe = mc.expert_ffn;
  c->Epad = (c->E + 127) / 128 * 128;

  const int64_t page_bytes_all = (int64_t)c->nl * c->hkv * kPage * c->hd * 2 * c->esz;
  const int64_t worst = (int64_t)c->P * c->pp + (int64_t)c->n_traj * ((c->cap + kPage - 1) / kPage);
  int64_t n_pages = worst;
  if (rc.kv_pool_bytes > 0) n_pages = std::min<int64_t>(worst, (int64_t)(rc.kv_pool_bytes / page_bytes_all));
  if (n_pages < (int64_t)c->P * c->pp || n_pages >= (1ll << 31)) { delete c; return DARTS_ENOMEM; }
  c->n_pages = n_pages;
  c->pool_layer_elems = n_pages * c->hkv * kPage * c->hd;

  size_t free_b = 0, total_b = 0;
  if (hipMemGetInfo(&free_b, &total_b) != hipSuccess) { delete c; return DARTS_EHIP; }
  if (mc.weights) {
    // every caller tensor must lie inside one device allocation of at least
    // its size, so the copy never reads past the caller's memory
    const int32_t nw = darts_weight_count(&mc);
    for (int32_t i = 0; i < nw; ++i) {
      void* base = nullptr;
      size_t size = 0;
      if (hipMemGetAddressRange(&base, &size, const_cast<void*>(mc.weights[i])) != hipSuccess ||
          (const char*)mc.weights[i] + caller_weight_bytes(mc, i) > (const char*)base + size) {
        (void)hipGetLastError();
        delete c;
        return DARTS_EINVAL;
      }
    }
  }
  const int rows_pf = c->P * c->Lp;
  const int rows_max = std::max(rows_pf, c->n_traj);
  const size_t ffn_elems = moe ? (size_t)c->E * c->d + (size_t)3 * c->E * c->Fe * c->d
                                : (size_t)3 * c->F * c->d;
  const size_t wbytes = ((size_t)c->V * c->d * 2 +
                         (size_t)c->nl * ((size_t)qkv_w * c->d + (size_t)c->d * c->hq * c->hd +
                                          ffn_elems)) * c->esz;
  const size_t poolb = (size_t)n_pages * page_bytes_all;
  // weights, the pool and the fp32 logits of a full batch (the largest
  // buffers; a failing allocation of the rest is reported the same way)
  const size_t logitb = (size_t)c->n_traj * c->V * 4;
  if (wbytes + poolb + logitb > free_b) { delete c; return DARTS_ENOMEM; }

  hipError_t e = hipSuccess;
  auto A = [&](auto** p, size_t bytes) { if (e == hipSuccess) e = dalloc(c, p, bytes); };
  A(&c->embed, (size_t)c->V * c->d * c->esz);
  A(&c->lm_head, (size_t)c->V * c->d * c->esz);
  c->layers.resize(c->nl);
  for (auto& w : c->layers) {
    A(&w.wqkv, (size_t)qkv_w * c->d * c->esz);
    A(&w.wo, (size_t)c->d * c->hq * c->hd * c->esz);
    if (moe) {
      A(&w.wrouter, (size_t)c->Epad * c->d * c->esz);
      A(&w.wegu, (size_t)c->E * 2 * c->Fe * c->d * c->esz);
      A(&w.wedown, (size_t)c->E * c->d * c->Fe * c->esz);
    } else {
      A(&w.wgu, (size_t)2 * c->F * c->d * c->esz);
      A(&w.wdown, (size_t)c->d * c->F * c->esz);
    }
  }
  A(&c->kpool, (size_t)c->nl * c->pool_layer_elems * c->esz);
  A(&c->vpool, (size_t)c->nl * c->pool_layer_elems * c->esz);
  const int max_pos = c->Lp + c->cap + 1;
  A(&c->rope, (size_t)max_pos * (c->hd / 2) * sizeof(float2));
  A(&c->page_table, (size_t)c->n_traj * c->max_pages * 4);
  A(&c->free_stack, (size_t)n_pages * 4);
  A(&c->dcnt, 64);
  A(&c->gen, (size_t)c->n_traj * 4);
  A(&c->sum_lp, (size_t)c->n_traj * 4);
  A(&c->status, (size_t)c->n_traj);
  A(&c->freed, (size_t)c->n_traj);
  A(&c->last_tok, (size_t)c->n_traj * 4);
  A(&c->forced_len, (size_t)c->n_traj * 4);
  A(&c->refcnt, (size_t)c->P * 4);
  A(&c->group_done, (size_t)c->P);
  A(&c->done_step, (size_t)c->P * 4);
  A(&c->kept, (size_t)c->P * k * 4);
  A(&c->live[0], (size_t)c->n_traj * 4);
  A(&c->live[1], (size_t)c->n_traj * 4);
  A(&c->grp_m, (size_t)c->P * 4);
  A(&c->grp_cnt, (size_t)c->P * 4);
  A(&c->grp_rel, (size_t)c->P * 4);
  A(&c->trj_cnt, (size_t)c->n_traj * 4);
  A(&c->prefill_pt, (size_t)rows_pf * 4);
  A(&c->last_rows, (size_t)c->P * 4);
  A(&c->x, (size_t)rows_max * c->d * 4);
  A(&c->xn, (size_t)rows_max * c->d * c->esz);
  A(&c->qkv, (size_t)rows_max * qkv_w * 4);
  A(&c->q, (size_t)rows_max * c->hq * c->hd * c->esz);
  A(&c->attn, (size_t)rows_max * c->hq * c->hd * c->esz);
  A(&c->hbuf, (size_t)rows_max * std::max(c->F, 1) * c->esz);
  if (moe) {
    const size_t pairs = (size_t)rows_max * c->topk;
    A(&c->m_topk_id, pairs * 4);
    A(&c->m_topk_w, pairs * 4);
    A(&c->m_pos_of, pairs * 4);
    A(&c->m_cnt, (size_t)3 * c->E * 4);
    A(&c->m_logits, (size_t)rows_max * c->Epad * 4);
    A(&c->m_mtiles, (pairs / kGroupedTileRowsMin + c->E + 1) * 4);
    A(&c->m_mtiles_dn, (pairs / kGroupedTileRowsMin + c->E + 1) * 4);
    A(&c->m_row_of, pairs * 4);
    A(&c->m_h_perm, pairs * c->Fe * 2);
    A(&c->m_y_perm, pairs * c->d * 2);
    A(&c->m_touched, (size_t)c->nl * 4);
  }
  if (rc.flags & DARTS_FLAG_STREAM) {
    A(&c->hist_tok, (size_t)c->n_traj * c->cap * 4);
    A(&c->hist_lp, (size_t)c->n_traj * c->cap * 4);
    A(&c->streamed, (size_t)c->n_traj * 4);
    A(&c->fin_sent, (size_t)c->n_traj);
    A(&c->stream_off, (size_t)c->n_traj * 4);
  }
  A(&c->xlast, (size_t)c->P * c->d * 4);
  A(&c->logits, (size_t)c->n_traj * c->V * 4);
  c->samp_part_cap = (int64_t)kSampleBlocks + c->n_traj;
  A(&c->samp_parts, (size_t)c->samp_part_cap * sizeof(SamplePart));
  c->gemm_ws_bytes = gemm_ws_need(c);
  A(&c->gemm_ws, c->gemm_ws_bytes);
  c->share_prefix = c->bf16 && c->m > 1 && c->pp > 0 && (c->rc.flags & DARTS_FLAG_SHARED_PREFIX);
  c->attn_ws_bytes = std::max(attn_workspace_bytes(c->n_traj, c->hq, c->hkv, c->hd, c->Lp + c->cap),
                              attn_workspace_bytes(rows_pf, c->hq, c->hkv, c->hd, c->Lp));
  if (c->share_prefix)
    c->attn_ws_bytes = std::max(c->attn_ws_bytes, attn_shared_workspace_bytes(c->n_traj, c->hq, c->hkv,
                                                                               c->hd, c->Lp + c->cap, c->pp));
  A(&c->attn_ws, c->attn_ws_bytes);
  if (e == hipSuccess) e = hipHostMalloc((void**)&c->h_info, 64, hipHostMallocDefault);
  if (e == hipSuccess && moe && (rc.flags & DARTS_FLAG_TIMING))
    e = hipHostMalloc((void**)&c->h_touched, (size_t)c->nl * 4, hipHostMallocDefault);
  if (e == hipSuccess && (rc.flags & DARTS_FLAG_STEP_TIMES)) {
    e = hipEventCreate(&c->step_ev[0]);
    if (e == hipSuccess) e = hipEventCreate(&c->step_ev[1]);
  }
  if (e != hipSuccess) {
    free_all(c);
    delete c;
    (void)hipGetLastError();
    return e == hipErrorOutOfMemory ? DARTS_ENOMEM : DARTS_EHIP;
  }
  // host-computed index tables (uploaded once)
  {
    std::vector<int32_t> pf(rows_pf), lr(c->P);
    for (int r = 0; r < rows_pf; ++r) pf[r] = (r / c->Lp) * c->m;
    for (int i = 0; i < c->P; ++i) lr[i] = i * c->Lp + c->Lp - 1;
    e = hipMemcpyAsync(c->prefill_pt, pf.data(), pf.size() * 4, hipMemcpyHostToDevice, c->st);
    if (e == hipSuccess) e = hipMemcpyAsync(c->last_rows, lr.data(), lr.size() * 4, hipMemcpyHostToDevice, c->st);
    if (e == hipSuccess) e = hipStreamSynchronize(c->st);
  }
  int rcode = DARTS_OK;
  if (e != hipSuccess) rcode = fail_hip(c, e, "upload index tables");
  if (rcode == DARTS_OK) rcode = c->mc.weights ? copy_weights(c) : init_weights(c);
  if (rcode == DARTS_OK && c->moe) rcode = pack_expert_weights(c);
  if (rcode == DARTS_OK) {
    e = launch_rope_table(c->rope, max_pos, c->hd, (double)mc.rope_theta, c->st);
    if (e == hipSuccess)
      e = launch_iota_perm(c->free_stack, n_pages, rc.page_perm_seed,
                           (rc.flags & DARTS_FLAG_PERMUTE_PAGES) != 0, c->st);
    const int32_t top = (int32_t)n_pages;
    if (e == hipSuccess) e = hipMemcpyAsync(c->dcnt, &top, 4, hipMemcpyHostToDevice, c->st);
    if (e == hipSuccess) e = hipMemsetAsync(c->gen, 0, (size_t)c->n_traj * 4, c->st);
    if (e == hipSuccess) e = hipMemsetAsync(c->sum_lp, 0, (size_t)c->n_traj * 4, c->st);
    if (e == hipSuccess) e = hipMemsetAsync(c->freed, 0, (size_t)c->n_traj, c->st);
    if (e == hipSuccess && c->streamed) e = hipMemsetAsync(c->streamed, 0, (size_t)c->n_traj * 4, c->st);
    if (e == hipSuccess && c->fin_sent) e = hipMemsetAsync(c->fin_sent, 0, (size_t)c->n_traj, c->st);
    if (e == hipSuccess) e = hipMemsetAsync(c->group_done, 0, (size_t)c->P, c->st);
    if (e == hipSuccess) e = hipMemsetAsync(c->kept, 0xff, (size_t)c->P * c->k * 4, c->st);
    if (e == hipSuccess) e = hipMemsetAsync(c->done_step, 0xff, (size_t)c->P * 4, c->st);
    if (e == hipSuccess) e = hipMemsetAsync(c->page_table, 0xff, (size_t)c->n_traj * c->max_pages * 4, c->st);
    if (e == hipSuccess) e = hipStreamSynchronize(c->st);
    c->plan.assign(c->P, c->m);
    if (e == hipSuccess) e = upload_plan(c);
    if (e != hipSuccess) rcode = fail_hip(c, e, "init");
  }
  if (rcode != DARTS_OK) {
    free_all(c);
    delete c;
    return rcode;
  }
  c->free_top = (int)n_pages;
  c->mc.weights = nullptr;   // the caller's array is not referenced after init
  *out = c;
  return DARTS_OK;
}

int darts_reset(darts_ctx* c) {
  if (!c) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  hipError_t e = hipStreamSynchronize(c->st);
  const int32_t top = (int32_t)c->n_pages;
  if (e == hipSuccess)
    e = launch_iota_perm(c->free_stack, c->n_pages, c->rc.page_perm_seed,
                         (c->rc.flags & DARTS_FLAG_PERMUTE_PAGES) != 0, c->st);
  if (e == hipSuccess) e = hipMemcpyAsync(c->dcnt, &top, 4, hipMemcpyHostToDevice, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->gen, 0, (size_t)c->n_traj * 4, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->sum_lp, 0, (size_t)c->n_traj * 4, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->freed, 0, (size_t)c->n_traj, c->st);
  if (e == hipSuccess && c->streamed) e = hipMemsetAsync(c->streamed, 0, (size_t)c->n_traj * 4, c->st);
  if (e == hipSuccess && c->fin_sent) e = hipMemsetAsync(c->fin_sent, 0, (size_t)c->n_traj, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->group_done, 0, (size_t)c->P, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->kept, 0xff, (size_t)c->P * c->k * 4, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->done_step, 0xff, (size_t)c->P * 4, c->st);
  if (e == hipSuccess) e = hipMemsetAsync(c->page_table, 0xff, (size_t)c->n_traj * c->max_pages * 4, c->st);
  if (e == hipSuccess) e = hipStreamSynchronize(c->st);
  c->plan.assign(c->P, c->m);
  if (e == hipSuccess) e = upload_plan(c);
  if (e != hipSuccess) return fail_hip(c, e, "reset");
  c->phase = 0; c->cur = 0; c->n_live = 0; c->n_done = 0; c->free_top = (int)c->n_pages;
  c->step = 0; c->tokens = 0; c->hwm = 0; c->last_rows_out = 0;
  c->pending.clear();
  c->step_rows = 0; c->st_rows.clear(); c->st_ms.clear(); c->prefill_ms = 0.f;
  c->attn_ms = c->attn_bytes = c->attn_traj_bytes = 0.0; c->attn_launches = 0;
  c->gemm_ms = c->gemm_flop = 0.0; c->gemm_launches = 0;
  for (int i = 0; i < 6; ++i) c->cls_ms[i] = c->cls_flop[i] = 0.0;
  for (int i = 0; i < 2; ++i) { c->moe_ms[i] = c->moe_bytes[i] = 0.0; c->moe_launches[i] = 0; }
  return DARTS_OK;
}

int darts_set_plan(darts_ctx* c, const int32_t* h_plan) {
  if (!c || !h_plan) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  if (c->phase != 0) return DARTS_ESTATE;
  for (int i = 0; i < c->P; ++i)
    if (h_plan[i] < c->k || h_plan[i] > c->m) return DARTS_EINVAL;
  c->plan.assign(h_plan, h_plan + c->P);
  hipError_t e = upload_plan(c);
  if (e != hipSuccess) return fail_hip(c, e, "set plan");
  return DARTS_OK;
}

int darts_destroy(darts_ctx* c) {
  if (!c) return DARTS_EINVAL;
  (void)hipStreamSynchronize(c->st);
  free_all(c);
  delete c;
  return DARTS_OK;
}

}  // extern "C"

// Attention with optional event timing.
static int run_attention(darts_ctx* c, int layer, int n_rows, const int32_t* row_pt, int ctx_mod,
                         int ctx_base, int max_ctx) {
  void* kp = (char*)c->kpool + (size_t)layer * c->pool_layer_elems * c->esz;
  void* vp = (char*)c->vpool + (size_t)layer * c->pool_layer_elems * c->esz;
  // algorithmic bytes: every distinct key and value once per kv head (with a
  // shared prefix, a prompt's prefix once per live group), q and out once,
  // one page id per 16 keys of each row
  const double ctx = ctx_base;
  const double kv_tok = (double)c->hkv * c->hd * 2.0 * c->esz;
  const double per_row_fixed = 2.0 * c->hq * c->hd * c->esz + std::ceil(ctx / kPage) * 4.0;
  const double traj_bytes = (double)n_rows * (ctx * kv_tok + per_row_fixed);
  const bool shared = c->share_prefix && ctx_mod == 0 && ctx_base > c->pp * kPage;
  double bytes = traj_bytes, grp_bytes = 0.0;
  if (shared) {
    bytes = (double)n_rows * ((ctx - c->pp * kPage) * kv_tok + per_row_fixed);
    grp_bytes = (double)c->pp * kPage * kv_tok;
  }
  // decode launches are timed around the attention kernels themselves (events
  // recorded inside the launcher)
  const int ti = ctx_mod == 0 ? treserve(c, 0, bytes) : -1;
  if (ti >= 0) { c->pending[ti].units_grp = grp_bytes; c->pending[ti].traj_units = traj_bytes; }
  hipEvent_t e0 = ti >= 0 ? c->events[2 * ti] : nullptr, e1 = ti >= 0 ? c->events[2 * ti + 1] : nullptr;
  if (shared) {
    HIPCHK(c, launch_attention_shared(c->q, kp, vp, c->n_pages, c->page_table, c->max_pages, row_pt,
                                      c->n_traj, c->m, c->pp, layer == 0, ctx_base, n_rows, c->hq,
                                      c->hkv, c->hd, c->attn,
                                      c->attn_ws, c->attn_ws_bytes, c->st, e0, e1, c->dcnt + 8));
    return DARTS_OK;
  }
  HIPCHK(c, launch_attention(c->q, kp, vp, c->n_pages, c->page_table, c->max_pages, row_pt, nullptr,
                             ctx_mod, ctx_base, n_rows, c->hq, c->hkv, c->hd, max_ctx, c->bf16,
                             c->attn, c->attn_ws, c->attn_ws_bytes, c->st, e0, e1));
  return DARTS_OK;
}

enum { G_QKV = 0, G_O, G_GU, G_DOWN, G_LM, G_MOE };
// TimedLaunch kinds of the grouped expert GEMMs (after the GEMM classes)
enum { kMoeGu = 1 + G_MOE + 1, kMoeDown = kMoeGu + 1 };
static hipError_t gemm_t(darts_ctx* c, int cls, const void* A, int lda, const void* W, int ldw,
                         void* C, int ldc, int M, int N, int K, int epi) {
  const int ti = tbegin(c, 1 + cls, 2.0 * M * N * K);
  hipError_t e = launch_gemm(c->bf16, A, lda, W, ldw, C, ldc, M, N, K, epi, c->gemm_ws,
                             c->gemm_ws_bytes, c->st);
  tend(c, ti);
  return e;
}

// x += A . W^T (residual projection), then xn = RMSNorm(x) when the two can
// be fused (bf16 dense models with a split-K plan): *normed reports it.
static hipError_t gemm_add_t(darts_ctx* c, int cls, const void* A, int lda, const void* W, int ldw,
                             int M, int K, bool* normed) {
  const int ti = tbegin(c, 1 + cls, 2.0 * M * c->d * K);
  hipError_t e;
  if (c->bf16) {
    e = launch_gemm_add_norm(A, lda, W, ldw, c->x, c->d, M, c->d, K, c->gemm_ws, c->gemm_ws_bytes,
                             c->mc.rms_eps, c->xn, c->st, normed);
  } else {
    *normed = false;
    e = launch_gemm(false, A, lda, W, ldw, c->x, c->d, M, c->d, K, EPI_ADD_F32, c->gemm_ws,
                    c->gemm_ws_bytes, c->st);
  }
  tend(c, ti);
  return e;
}

// Decoder layers over n rows whose residual stream is in c->x.  normed: c->xn
// already holds RMSNorm(x) on entry; on return, whether it holds the final
// residual's norm.
static int run_layers(darts_ctx* c, int n, const int32_t* row_pt, const int32_t* row_key, int pos_mod,
                      int pos_base, int ctx_mod, int ctx_base, int max_ctx, bool* normed) {
  const bool b = c->bf16;
  const int d = c->d, hqd = c->hq * c->hd;
  for (int l = 0; l < c->nl; ++l) {
    LayerW& w = c->layers[l];
    void* kp = (char*)c->kpool + (size_t)l * c->pool_layer_elems * c->esz;
    void* vp = (char*)c->vpool + (size_t)l * c->pool_layer_elems * c->esz;
    if (!*normed) HIPCHK(c, launch_rmsnorm(c->x, n, d, c->mc.rms_eps, c->xn, b, c->st));
    // QKV projection; with a split-K plan the partial sums go straight to the
    // RoPE + KV-append kernel, which adds them
    int n_split = 1;
    const float* qkv_src = c->qkv;
    if (b) {
      const int ti = tbegin(c, 1 + G_QKV, 2.0 * n * c->qkv_w * d);
      HIPCHK(c, launch_gemm_f32_or_partials(c->xn, d, w.wqkv, d, c->qkv, c->qkv_w, n, c->qkv_w, d,
                                            c->gemm_ws, c->gemm_ws_bytes, c->st, &n_split));
      tend(c, ti);
      if (n_split > 1) qkv_src = (const float*)c->gemm_ws;
    } else {
      HIPCHK(c, gemm_t(c, G_QKV, c->xn, d, w.wqkv, d, c->qkv, c->qkv_w, n, c->qkv_w, d, EPI_F32));
    }
    HIPCHK(c, launch_rope_append2(qkv_src, n_split, (int64_t)n * c->qkv_w, n, c->hq, c->hkv, c->hd,
                                  row_pt, pos_mod, pos_base, c->page_table, c->max_pages,
                                  c->n_pages, c->rope, c->q, kp, vp, b, c->st));
    int r = run_attention(c, l, n, row_pt, ctx_mod, ctx_base, max_ctx);
    if (r != DARTS_OK) return r;
    HIPCHK(c, gemm_add_t(c, G_O, c->attn, hqd, w.wo, hqd, n, hqd, normed));
    if (!*normed) HIPCHK(c, launch_rmsnorm(c->x, n, d, c->mc.rms_eps, c->xn, b, c->st));
    if (c->moe) {
      MoeArgs m{};   // every optional pointer and event NULL unless set below
      m.xn = (bf16_t*)c->xn; m.x = c->x; m.n_rows = n; m.d = d; m.E = c->E; m.k = c->topk;
      m.eps = c->mc.rms_eps; m.row_of = c->m_row_of;
      m.Fe = c->Fe; m.w_router = (const bf16_t*)w.wrouter; m.w_gu = (const bf16_t*)w.wegu;
      m.E_pad = c->Epad; m.logits = c->m_logits; m.gemm_ws = c->gemm_ws;
      m.n_mtiles = c->m_mtiles; m.mtiles = c->m_mtiles + 1;
      m.n_mtiles_dn = c->m_mtiles_dn; m.mtiles_dn = c->m_mtiles_dn + 1;
      m.gemm_ws_bytes = c->gemm_ws_bytes;
      m.w_down = (const bf16_t*)w.wedown; m.topk_id = c->m_topk_id; m.topk_w = c->m_topk_w;
      m.pos_of = c->m_pos_of; m.counts = c->m_cnt; m.offsets = c->m_cnt + c->E;
      m.cursors = c->m_cnt + 2 * c->E;
      m.h_perm = (bf16_t*)c->m_h_perm; m.y_perm = (bf16_t*)c->m_y_perm;
      const int64_t dstride = (int64_t)c->nl * c->topk;
      m.route_key = row_key; m.dbg_stride = dstride;
      m.force_ids = c->dbg_force_ids ? c->dbg_force_ids + (int64_t)l * c->topk : nullptr;
      m.own_ids_out = c->dbg_own_ids ? c->dbg_own_ids + (int64_t)l * c->topk : nullptr;
      m.used_p_out = c->dbg_used_p ? c->dbg_used_p + (int64_t)l * c->topk : nullptr;
      const double flop = 2.0 * n * ((double)c->E * d + (double)c->topk * 3.0 * c->Fe * d);
      const int ti = tbegin(c, 1 + G_MOE, flop);
      if (ti >= 0) {
        // the two grouped expert GEMMs inside the block are timed on their
        // own; their bytes follow from the touched-expert count read back
        // after the step
        const int tg = treserve(c, kMoeGu, 0.0), td = treserve(c, kMoeDown, 0.0);
        if (tg >= 0 && td >= 0) {
          m.ev_gu0 = c->events[2 * tg]; m.ev_gu1 = c->events[2 * tg + 1];
          m.ev_down0 = c->events[2 * td]; m.ev_down1 = c->events[2 * td + 1];
          m.touched_out = c->m_touched + l;
          c->pending[tg].touched_slot = c->pending[td].touched_slot = l;
          c->pending[tg].rows = c->pending[td].rows = (double)n * c->topk;
        }
      }
      HIPCHK(c, launch_moe_ffn(m, c->st, normed));
      tend(c, ti);
      continue;
    }
    HIPCHK(c, gemm_t(c, G_GU, c->xn, d, w.wgu, d, c->hbuf, c->F, n, 2 * c->F, d, EPI_SWIGLU));
    HIPCHK(c, gemm_add_t(c, G_DOWN, c->hbuf, c->F, w.wdown, c->F, n, c->F, normed));
  }
  return DARTS_OK;
}

static int write_out_rows(darts_ctx* c, darts_step_out* out, int n) {
  if (out) out->n_rows = n;
  c->last_rows_out = n;
  return DARTS_OK;
}

extern "C" {

int darts_prefill(darts_ctx* c, const int32_t* d_prompts, const int32_t* d_forced_len,
                  const int32_t* d_force_tokens, darts_step_out* out) {
  if (!c || !d_prompts || !d_forced_len || !out) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  if (c->phase != 0) return DARTS_ESTATE;
  if (!out->traj_id || !out->token || !out->logprob || !out->entropy || !out->finished)
    return DARTS_EINVAL;
  const bool b = c->bf16;
  c->timed_weight = timing_on(c) ? 1.0 : 0.0;
  const int rows = c->P * c->Lp;
  HIPCHK(c, step_begin(c, -1));
  HIPCHK(c, hipMemcpyAsync(c->forced_len, d_forced_len, (size_t)c->n_traj * 4,
                           hipMemcpyDeviceToDevice, c->st));
  HIPCHK(c, launch_prefill_pages(c->P, c->m, c->grp_m, c->pp, c->page_table, c->max_pages,
                                 c->free_stack, c->dcnt, c->refcnt, c->st));
  bool normed = b;
  if (b) HIPCHK(c, launch_embed_norm(c->embed, d_prompts, nullptr, rows, c->d, c->V, c->mc.rms_eps,
                                     c->x, c->xn, c->st));
  else HIPCHK(c, launch_embed_v(c->embed, b, d_prompts, nullptr, rows, c->d, c->V, c->x, c->st));
  int r = run_layers(c, rows, c->prefill_pt, nullptr, c->Lp, 0, c->Lp, 1, c->Lp, &normed);
  if (r != DARTS_OK) return r;
  HIPCHK(c, launch_gather_rows(c->x, c->last_rows, c->P, c->d, c->xlast, c->st));
  HIPCHK(c, launch_rmsnorm(c->xlast, c->P, c->d, c->mc.rms_eps, c->xn, b, c->st));
  HIPCHK(c, launch_gemm(b, c->xn, c->d, c->lm_head, c->d, c->logits, c->V, c->P, c->V, c->d,
                        EPI_F32, c->gemm_ws, c->gemm_ws_bytes, c->st));
  SampleArgs a{};
  a.logits = c->logits; a.n_rows = c->n_start; a.vocab = c->V; a.bf16 = false;
  a.seed = c->rc.sample_seed; a.temperature = c->rc.temperature; a.traj_base = c->rc.traj_base;
  a.row_logit = nullptr; a.logit_div = c->m;
  a.traj = c->live[c->cur]; a.step = nullptr; a.force = d_force_tokens;
  a.token_out = out->token; a.sampled_out = out->sampled; a.logprob_out = out->logprob;
  a.entropy_out = out->entropy; a.gen = c->gen; a.sum_lp = c->sum_lp; a.status = c->status;
  a.last_tok = c->last_tok; a.forced_len = c->forced_len; a.finished_out = out->finished;
  a.traj_out = out->traj_id; a.cap = c->cap; a.eos = c->V - 1;
  a.hist_tok = c->hist_tok; a.hist_lp = c->hist_lp;
  a.part_out = c->samp_parts; a.part_cap = c->samp_part_cap;
  HIPCHK(c, launch_sample(a, c->st));
  c->free_top -= c->P * c->pp;
  c->hwm = std::max<int64_t>(c->hwm, c->n_pages - c->free_top);
  c->phase = 1;
  c->step = 1;
  c->n_live = c->n_start;
  c->tokens += c->n_start;
  HIPCHK(c, hipStreamSynchronize(c->st));
  return write_out_rows(c, out, c->n_start);
}

int darts_decode_step(darts_ctx* c, const int32_t* d_force_tokens, darts_step_out* out) {
  if (!c || !out) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  if (c->phase != 1 || c->n_live <= 0) return DARTS_ESTATE;
  if (!out->traj_id || !out->token || !out->logprob || !out->entropy || !out->finished)
    return DARTS_EINVAL;
  const bool b = c->bf16;
  const int n = c->n_live;
  const int64_t s_before = c->step;               // tokens generated so far by every live row
  const int pos = c->Lp + (int)s_before - 1;      // position of the token consumed now
  if (pos + 1 > c->Lp + c->cap) return DARTS_ESTATE;
  const bool need_pages = ((s_before - 1) % kPage) == 0;
  if (need_pages && n > c->free_top) return DARTS_ENOMEM;
  c->timed_weight = (timing_on(c) && s_before % kTimingStride == 0) ? (double)kTimingStride : 0.0;
  HIPCHK(c, step_begin(c, n));
  int32_t* live = c->live[c->cur];
  if (need_pages) {
    HIPCHK(c, launch_alloc_pages(live, n, c->gen, c->pp, c->page_table, c->max_pages, c->free_stack,
                                 c->dcnt, c->dcnt + 4, c->st));
    c->free_top -= n;
    c->hwm = std::max<int64_t>(c->hwm, c->n_pages - c->free_top);
  }
  bool normed = b;
  if (b) HIPCHK(c, launch_embed_norm(c->embed, c->last_tok, live, n, c->d, c->V, c->mc.rms_eps, c->x,
                                     c->xn, c->st));
  else HIPCHK(c, launch_embed_v(c->embed, b, c->last_tok, live, n, c->d, c->V, c->x, c->st));
  int r = run_layers(c, n, live, live, 0, pos, 0, pos + 1, pos + 1, &normed);
  if (r != DARTS_OK) return r;
  if (!normed) HIPCHK(c, launch_rmsnorm(c->x, n, c->d, c->mc.rms_eps, c->xn, b, c->st));
  HIPCHK(c, gemm_t(c, G_LM, c->xn, c->d, c->lm_head, c->d, c->logits, c->V, n, c->V, c->d, EPI_F32));
  SampleArgs a{};
  a.logits = c->logits; a.n_rows = n; a.vocab = c->V; a.bf16 = false;
  a.seed = c->rc.sample_seed; a.temperature = c->rc.temperature; a.traj_base = c->rc.traj_base;
  a.row_logit = nullptr; a.logit_div = 0;
  a.traj = live; a.step = nullptr; a.force = d_force_tokens;
  a.token_out = out->token; a.sampled_out = out->sampled; a.logprob_out = out->logprob;
  a.entropy_out = out->entropy; a.gen = c->gen; a.sum_lp = c->sum_lp; a.status = c->status;
  a.last_tok = c->last_tok; a.forced_len = c->forced_len; a.finished_out = out->finished;
  a.traj_out = out->traj_id; a.cap = c->cap; a.eos = c->V - 1;
  a.hist_tok = c->hist_tok; a.hist_lp = c->hist_lp;
  a.part_out = c->samp_parts; a.part_cap = c->samp_part_cap;
  HIPCHK(c, launch_sample(a, c->st));
  c->step += 1;
  c->tokens += n;
  return write_out_rows(c, out, n);
}

int darts_select_and_prune(darts_ctx* c, int32_t* d_kept, int32_t* d_done_step, int32_t* h_n_live,
                           int32_t* h_n_done) {
  if (!c) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  if (c->phase == 0) return DARTS_ESTATE;
  PruneArgs a{};
  a.status = c->status; a.gen = c->gen; a.sum_lp = c->sum_lp; a.freed = c->freed;
  a.refcnt = c->refcnt; a.group_done = c->group_done; a.done_step = c->done_step; a.kept = c->kept;
  a.n_groups = c->P; a.m = c->m; a.k = c->k; a.L = c->L; a.m_up = c->m_up; a.grp_m = c->grp_m;
  a.early_stop = (c->rc.flags & DARTS_FLAG_NO_ABORT) ? 0 : 1;
  a.step = (int)c->step;
  a.page_table = c->page_table; a.pt_stride = c->max_pages; a.prompt_pages = c->pp;
  a.free_stack = c->free_stack; a.free_top = c->dcnt; a.n_pages = (int)c->n_pages;
  a.grp_cnt = c->grp_cnt; a.grp_rel = c->grp_rel; a.trj_cnt = c->trj_cnt;
  a.live_in = c->live[c->cur]; a.n_live_in = c->n_live; a.live_out = c->live[c->cur ^ 1];
  a.info = c->dcnt + 4;
  HIPCHK(c, launch_prune(a, c->st));
  if (d_kept)
    HIPCHK(c, hipMemcpyAsync(d_kept, c->kept, (size_t)c->P * c->k * 4, hipMemcpyDeviceToDevice, c->st));
  if (d_done_step)
    HIPCHK(c, hipMemcpyAsync(d_done_step, c->done_step, (size_t)c->P * 4, hipMemcpyDeviceToDevice, c->st));
  const int timed_rows = c->step_rows;
  if (timed_rows != 0) HIPCHK(c, hipEventRecord(c->step_ev[1], c->st));
  HIPCHK(c, hipMemcpyAsync(c->h_info, c->dcnt + 4, 32, hipMemcpyDeviceToHost, c->st));
  bool touched = false;
  for (const TimedLaunch& t : c->pending) touched = touched || t.touched_slot >= 0;
  if (touched && c->h_touched)
    HIPCHK(c, hipMemcpyAsync(c->h_touched, c->m_touched, (size_t)c->nl * 4, hipMemcpyDeviceToHost, c->st));
  HIPCHK(c, hipStreamSynchronize(c->st));
  if (timed_rows != 0) {
    float ms = 0.f;
    HIPCHK(c, hipEventElapsedTime(&ms, c->step_ev[0], c->step_ev[1]));
    if (timed_rows < 0) c->prefill_ms += ms;
    else { c->st_rows.push_back(timed_rows); c->st_ms.push_back(ms); }
    c->step_rows = 0;
  }
  c->cur ^= 1;
  c->n_live = c->h_info[0];
  c->n_done = c->h_info[1];
  c->free_top = c->h_info[2];
  if (c->n_done == c->P) c->phase = 2;
  for (size_t i = 0; i < c->pending.size(); ++i) {
    float ms = 0.f;
    HIPCHK(c, hipEventElapsedTime(&ms, c->events[2 * i], c->events[2 * i + 1]));
    const TimedLaunch& t = c->pending[i];
    const double w = t.weight;
    if (t.kind == 0) {
      // h_info[4]: live prompt groups of the step (written by the shared-prefix launch)
      const double units = t.units + (t.units_grp > 0.0 ? t.units_grp * c->h_info[4] : 0.0);
      c->attn_ms += w * ms; c->attn_bytes += w * units; c->attn_traj_bytes += w * t.traj_units;
      c->attn_launches += (int64_t)w;
    } else if (t.kind == kMoeGu || t.kind == kMoeDown) {
      // algorithmic bytes: the touched experts' weights once, the routed
      // rows' inputs and outputs (gate/up: bf16 rows in, bf16 SwiGLU rows out;
      // down: bf16 rows in, bf16 rows out)
      if (!c->h_touched || t.touched_slot < 0) continue;
      const double ne = c->h_touched[t.touched_slot];
      const double dd = c->d, fe = c->Fe;
      const int i = t.kind == kMoeGu ? 0 : 1;
      const double bytes = i == 0 ? ne * 2.0 * fe * dd * 2.0 + t.rows * (dd * 2.0 + fe * 2.0)
                                  : ne * dd * fe * 2.0 + t.rows * (fe * 2.0 + dd * 2.0);
      c->moe_ms[i] += w * ms; c->moe_bytes[i] += w * bytes; c->moe_launches[i] += (int64_t)w;
    } else {
      c->gemm_ms += w * ms; c->gemm_flop += w * t.units; c->gemm_launches += (int64_t)w;
      c->cls_ms[t.kind - 1] += w * ms; c->cls_flop[t.kind - 1] += w * t.units;
    }
  }
  c->pending.clear();
  if (h_n_live) *h_n_live = c->n_live;
  if (h_n_done) *h_n_done = c->n_done;
  return DARTS_OK;
}

int darts_get_stats(const darts_ctx* c, darts_stats* s) {
  if (!c || !s) return DARTS_EINVAL;
  s->steps = c->step;
  s->tokens_decoded = c->tokens;
  s->n_pages = c->n_pages;
  s->pages_used = c->n_pages - c->free_top;
  s->pages_hwm = c->hwm;
  s->n_live = c->n_live;
  s->n_done = c->n_done;
  s->attn_ms = c->attn_ms;
  s->attn_bytes = c->attn_bytes;
  s->attn_traj_bytes = c->attn_traj_bytes;
  s->attn_launches = c->attn_launches;
  s->gemm_ms = c->gemm_ms;
  s->gemm_flop = c->gemm_flop;
  s->gemm_launches = c->gemm_launches;
  for (int i = 0; i < 6; ++i) { s->gemm_cls_ms[i] = c->cls_ms[i]; s->gemm_cls_flop[i] = c->cls_flop[i]; }
  for (int i = 0; i < 2; ++i) {
    s->moe_expert_ms[i] = c->moe_ms[i];
    s->moe_expert_bytes[i] = c->moe_bytes[i];
    s->moe_expert_launches[i] = c->moe_launches[i];
  }
  return DARTS_OK;
}

int darts_get_step_times(const darts_ctx* c, int32_t* h_rows, float* h_ms, int32_t cap, int32_t* h_n,
                         float* h_prefill_ms) {
  if (!c || !h_n || cap < 0 || (cap > 0 && (!h_rows || !h_ms))) return DARTS_EINVAL;
  if (!step_times_on(c)) return DARTS_ESTATE;
  const int32_t n = (int32_t)c->st_ms.size();
  *h_n = n;
  for (int32_t i = 0; i < std::min(n, cap); ++i) { h_rows[i] = c->st_rows[i]; h_ms[i] = c->st_ms[i]; }
  if (h_prefill_ms) *h_prefill_ms = c->prefill_ms;
  return DARTS_OK;
}

int darts_stream_chunks(darts_ctx* c, int64_t threshold, int32_t flush, int32_t* d_desc,
                        int32_t* d_tokens, float* d_logprobs, int64_t out_cap, int32_t* h_n_desc,
                        int64_t* h_n_tokens) {
  if (!c || !d_desc || !h_n_desc || threshold < 1 || out_cap < 0) return DARTS_EINVAL;
  if (out_cap > 0 && (!d_tokens || !d_logprobs)) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  if (!c->hist_tok || c->phase == 0) return DARTS_ESTATE;
  StreamArgs a{};
  a.gen = c->gen; a.status = c->status; a.streamed = c->streamed; a.fin_sent = c->fin_sent;
  a.hist_tok = c->hist_tok; a.hist_lp = c->hist_lp; a.cap = c->cap; a.n_traj = c->n_traj;
  a.threshold = threshold; a.flush = flush ? 1 : 0; a.desc = d_desc; a.off = c->stream_off;
  a.tok_out = d_tokens; a.lp_out = d_logprobs; a.out_cap = out_cap; a.info = c->dcnt + 12;
  HIPCHK(c, launch_stream(a, c->st));
  HIPCHK(c, hipMemcpyAsync(c->h_info + 8, c->dcnt + 12, 8, hipMemcpyDeviceToHost, c->st));
  HIPCHK(c, hipStreamSynchronize(c->st));
  if (c->h_info[8] < 0) return DARTS_ENOMEM;
  *h_n_desc = c->h_info[8];
  if (h_n_tokens) *h_n_tokens = c->h_info[9];
  return DARTS_OK;
}

int darts_get_traj_scores(darts_ctx* c, int32_t* d_len, float* d_sum_lp, float* d_mean_lp,
                          uint8_t* d_status) {
  if (!c) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  if (d_len) HIPCHK(c, hipMemcpyAsync(d_len, c->gen, (size_t)c->n_traj * 4, hipMemcpyDeviceToDevice, c->st));
  if (d_sum_lp)
    HIPCHK(c, hipMemcpyAsync(d_sum_lp, c->sum_lp, (size_t)c->n_traj * 4, hipMemcpyDeviceToDevice, c->st));
  if (d_status)
    HIPCHK(c, hipMemcpyAsync(d_status, c->status, (size_t)c->n_traj, hipMemcpyDeviceToDevice, c->st));
  if (d_mean_lp) {
    // mean = fl32(sum / len), computed on the host copy to keep the device path small
    std::vector<float> s(c->n_traj), mlp(c->n_traj);
    std::vector<int32_t> ln(c->n_traj);
    HIPCHK(c, hipMemcpyAsync(s.data(), c->sum_lp, (size_t)c->n_traj * 4, hipMemcpyDeviceToHost, c->st));
    HIPCHK(c, hipMemcpyAsync(ln.data(), c->gen, (size_t)c->n_traj * 4, hipMemcpyDeviceToHost, c->st));
    HIPCHK(c, hipStreamSynchronize(c->st));
    for (int g = 0; g < c->n_traj; ++g) mlp[g] = ln[g] > 0 ? s[g] / (float)ln[g] : 0.f;
    HIPCHK(c, hipMemcpyAsync(d_mean_lp, mlp.data(), (size_t)c->n_traj * 4, hipMemcpyHostToDevice, c->st));
  }
  HIPCHK(c, hipStreamSynchronize(c->st));
  return DARTS_OK;
}

int darts_debug_logits(darts_ctx* c, float* d_dst, int32_t* h_n_rows) {
  if (!c || !d_dst) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  const int rows = c->phase == 1 && c->step == 1 ? c->P : c->last_rows_out;
  HIPCHK(c, hipMemcpyAsync(d_dst, c->logits, (size_t)rows * c->V * 4, hipMemcpyDeviceToDevice, c->st));
  HIPCHK(c, hipStreamSynchronize(c->st));
  if (h_n_rows) *h_n_rows = rows;
  return DARTS_OK;
}

int darts_debug_fill_kv(darts_ctx* c, int32_t byte) {
  if (!c || byte < 0 || byte > 255) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  if (c->phase != 0) return DARTS_ESTATE;
  const size_t bytes = (size_t)c->nl * c->pool_layer_elems * c->esz;
  HIPCHK(c, hipMemsetAsync(c->kpool, byte, bytes, c->st));
  HIPCHK(c, hipMemsetAsync(c->vpool, byte, bytes, c->st));
  HIPCHK(c, hipStreamSynchronize(c->st));
  return DARTS_OK;
}

int darts_debug_moe_routing(darts_ctx* c, const int32_t* d_force_ids, int32_t* d_own_ids,
                            float* d_used_p, int64_t n_keys) {
  if (!c) return DARTS_EINVAL;
  if (c->poisoned) return DARTS_EHIP;
  if (!c->moe) return DARTS_EINVAL;
  const bool any = d_force_ids || d_own_ids || d_used_p;
  if (any && n_keys < std::max<int64_t>((int64_t)c->P * c->Lp, c->n_traj)) return DARTS_EINVAL;
  c->dbg_force_ids = d_force_ids;
  c->dbg_own_ids = d_own_ids;
  c->dbg_used_p = d_used_p;
  return DARTS_OK;
}

// ------------------------------------------------------------- stateless

int darts_fill_uniform(void* d_dst, uint64_t n, int32_t tensor, uint64_t seed, int32_t dtype,
                       void* stream) {
  if ((!d_dst && n) || (dtype != DARTS_F32 && dtype != DARTS_BF16)) return DARTS_EINVAL;
  hipError_t e = launch_fill_uniform(d_dst, n, (uint32_t)tensor, seed, dtype == DARTS_BF16,
                                     (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

int darts_stream_read(const void* d_src, int64_t bytes, float* d_sink, void* stream) {
  if (bytes < 0 || bytes % 16) return DARTS_EINVAL;
  if (bytes == 0) return DARTS_OK;
  if (!d_src || ((uintptr_t)d_src & 15) || !d_sink) return DARTS_EINVAL;
  hipError_t e = launch_stream_read(d_src, bytes / 16, d_sink, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

int darts_fill_kv_pool(void* d_k_pool, void* d_v_pool, int64_t n_pages, int32_t n_kv_heads,
                       int32_t head_dim, uint64_t seed, int32_t dtype, void* stream) {
  if (!d_k_pool || !d_v_pool || n_pages < 1 || n_kv_heads < 1 || head_dim < 32 || head_dim % 32)
    return DARTS_EINVAL;
  if (dtype != DARTS_F32 && dtype != DARTS_BF16) return DARTS_EINVAL;
  hipError_t e = launch_fill_kv_pool(d_k_pool, d_v_pool, n_pages, n_kv_heads, head_dim, seed,
                                     dtype == DARTS_BF16, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

size_t darts_attn_workspace_bytes(int32_t n_rows, int32_t n_q_heads, int32_t n_kv_heads,
                                  int32_t head_dim, int32_t max_ctx) {
  if (n_rows < 1 || n_q_heads < 1 || n_kv_heads < 1 || max_ctx < 1) return 0;
  return attn_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim, max_ctx);
}

int darts_attn_decode(const void* d_q, const void* d_k_pool, const void* d_v_pool,
                           int64_t n_pages, const int32_t* d_page_table, int32_t pt_stride,
                           const int32_t* d_ctx_len, int32_t n_rows, int32_t n_q_heads,
                           int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx, int32_t dtype,
                           void* d_out, void* d_workspace, size_t workspace_bytes, void* stream) {
  if (n_rows < 0 || n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads ||
      n_q_heads / n_kv_heads > 16 || max_ctx < 1 || n_pages < 1)
    return DARTS_EINVAL;
  if (!(head_dim == 32 || head_dim == 64 || head_dim == 128)) return DARTS_EINVAL;
  if (dtype != DARTS_F32 && dtype != DARTS_BF16) return DARTS_EINVAL;
  if (pt_stride < (max_ctx + kPage - 1) / kPage) return DARTS_EINVAL;
  if (n_rows == 0) return DARTS_OK;
  if (!d_q || !d_k_pool || !d_v_pool || !d_page_table || !d_out) return DARTS_EINVAL;
  if (workspace_bytes < attn_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim, max_ctx))
    return DARTS_EINVAL;
  // no per-row contexts: every row attends to max_ctx keys (the equal-context
  // form of a decode step)
  hipError_t e = launch_attention(d_q, d_k_pool, d_v_pool, n_pages, d_page_table, pt_stride, nullptr,
                                  d_ctx_len, 0, d_ctx_len ? 0 : max_ctx, n_rows, n_q_heads, n_kv_heads,
                                  head_dim, max_ctx,
                                  dtype == DARTS_BF16, d_out, d_workspace, workspace_bytes,
                                  (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

}  // extern "C"

// Workspace of darts_attn_decode_noalloc: a fixed array in this library's code
// object, one copy per GPU (the runtime places it when the code object is
// loaded on that device).  Host code never uses the array's name as an
// address: the device address is looked up once per device with
// hipGetSymbolAddress and kept in g_scratch_ptr.  No call reads what an
// earlier call left in it (the attention kernels write every workspace entry
// they read within the same call), so nothing needs clearing between calls.
static __device__ __align__(256) unsigned char scratch[DARTS_ATTN_NOALLOC_SCRATCH_BYTES];
constexpr int kMaxScratchDevices = 64;
static std::mutex g_scratch_mu;
static void* g_scratch_ptr[kMaxScratchDevices] = {};

static hipError_t scratch_on_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxScratchDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return hipSuccess;
}

extern "C" {

int darts_attn_decode_noalloc(const void* d_q, const void* d_k_pool, const void* d_v_pool,
                              int64_t n_pages, const int32_t* d_page_table, int32_t pt_stride,
                              const int32_t* d_ctx_len, int32_t n_rows, int32_t n_q_heads,
                              int32_t n_kv_heads, int32_t head_dim, int32_t max_ctx, int32_t dtype,
                              void* d_out, void* stream) {
  if (n_rows < 0 || n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads ||
      n_q_heads / n_kv_heads > 16 || max_ctx < 1 || n_pages < 1)
    return DARTS_EINVAL;
  if (!(head_dim == 32 || head_dim == 64 || head_dim == 128)) return DARTS_EINVAL;
  if (dtype != DARTS_F32 && dtype != DARTS_BF16) return DARTS_EINVAL;
  if (pt_stride < (max_ctx + kPage - 1) / kPage) return DARTS_EINVAL;
  if (n_rows == 0) return DARTS_OK;
  if (!d_q || !d_k_pool || !d_v_pool || !d_page_table || !d_out) return DARTS_EINVAL;
  if (attn_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim, max_ctx) >
      (size_t)DARTS_ATTN_NOALLOC_SCRATCH_BYTES)
    return DARTS_EINVAL;
  void* ws = nullptr;
  if (scratch_on_current_device(&ws) != hipSuccess) return DARTS_EHIP;
  hipError_t e = launch_attention(d_q, d_k_pool, d_v_pool, n_pages, d_page_table, pt_stride, nullptr,
                                  d_ctx_len, 0, d_ctx_len ? 0 : max_ctx, n_rows, n_q_heads, n_kv_heads,
                                  head_dim, max_ctx, dtype == DARTS_BF16, d_out, ws,
                                  (size_t)DARTS_ATTN_NOALLOC_SCRATCH_BYTES, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

size_t darts_attn_shared_workspace_bytes(int32_t n_rows, int32_t n_q_heads, int32_t n_kv_heads,
                                         int32_t head_dim, int32_t ctx_len, int32_t prefix_pages) {
  if (n_rows < 1 || n_q_heads < 1 || n_kv_heads < 1 || ctx_len < 1 || prefix_pages < 1) return 0;
  return attn_shared_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim, ctx_len, prefix_pages);
}

int darts_attn_decode_shared(const void* d_q, const void* d_k_pool, const void* d_v_pool,
                             int64_t n_pages, const int32_t* d_page_table, int32_t pt_stride,
                             int32_t pt_rows, const int32_t* d_row_traj, int32_t m,
                             int32_t prefix_pages, int32_t ctx_len, int32_t n_rows, int32_t n_q_heads,
                             int32_t n_kv_heads, int32_t head_dim, int32_t dtype, void* d_out,
                             void* d_workspace, size_t workspace_bytes, void* stream) {
  if (n_rows < 0 || n_q_heads < 1 || n_kv_heads < 1 || n_q_heads % n_kv_heads ||
      n_q_heads / n_kv_heads > 16 || n_pages < 1 || pt_rows < 1 || m < 1 || prefix_pages < 1)
    return DARTS_EINVAL;
  if (!(head_dim == 32 || head_dim == 64 || head_dim == 128)) return DARTS_EINVAL;
  if (dtype != DARTS_BF16) return DARTS_EINVAL;
  if (ctx_len <= prefix_pages * kPage || pt_stride < (ctx_len + kPage - 1) / kPage) return DARTS_EINVAL;
  if (n_rows == 0) return DARTS_OK;
  if (!d_q || !d_k_pool || !d_v_pool || !d_page_table || !d_row_traj || !d_out) return DARTS_EINVAL;
  if (workspace_bytes <
      attn_shared_workspace_bytes(n_rows, n_q_heads, n_kv_heads, head_dim, ctx_len, prefix_pages))
    return DARTS_EINVAL;
  hipError_t e = launch_attention_shared(d_q, d_k_pool, d_v_pool, n_pages, d_page_table, pt_stride,
                                         d_row_traj, pt_rows, m, prefix_pages, true, ctx_len, n_rows,
                                         n_q_heads, n_kv_heads, head_dim, d_out, d_workspace,
                                         workspace_bytes, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

int darts_sample(const void* d_logits, int32_t n_rows, int32_t vocab, int32_t dtype, uint64_t seed,
                 const int32_t* d_traj, const int32_t* d_step, float temperature,
                 const int32_t* d_force, int32_t* d_token, float* d_logprob, float* d_entropy,
                 void* stream) {
  if (n_rows < 0 || vocab < 4 || vocab % 4 || !(temperature > 0.f)) return DARTS_EINVAL;
  if (dtype != DARTS_F32 && dtype != DARTS_BF16) return DARTS_EINVAL;
  if (n_rows == 0) return DARTS_OK;
  if (!d_logits || !d_traj || !d_step) return DARTS_EINVAL;
  SampleArgs a{};
  a.logits = d_logits; a.n_rows = n_rows; a.vocab = vocab; a.bf16 = dtype == DARTS_BF16;
  a.seed = seed; a.temperature = temperature; a.traj = d_traj; a.step = d_step; a.force = d_force;
  a.token_out = d_token; a.logprob_out = d_logprob; a.entropy_out = d_entropy;
  hipError_t e = launch_sample(a, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

size_t darts_gemm_workspace_bytes(int32_t M, int32_t N, int32_t K) {
  if (M < 1 || N < 1 || K < 1) return 0;
  return gemm_workspace_bytes(M, N, K);
}

int darts_gemm(const void* d_a, const void* d_w, void* d_c, int32_t M, int32_t N, int32_t K,
               int32_t dtype, int32_t epilogue, void* d_workspace, size_t workspace_bytes,
               void* stream) {
  if (M < 0 || N < 1 || K < 1) return DARTS_EINVAL;
  if (dtype != DARTS_F32 && dtype != DARTS_BF16) return DARTS_EINVAL;
  if (epilogue < 0 || epilogue > 3) return DARTS_EINVAL;
  if (epilogue == 3 && N % 32) return DARTS_EINVAL;
  if (dtype == DARTS_BF16 && (N % 128 || K % 256)) return DARTS_EINVAL;
  if (M == 0) return DARTS_OK;
  if (!d_a || !d_w || !d_c) return DARTS_EINVAL;
  const int ldc = epilogue == 3 ? N / 2 : N;
  const size_t need = dtype == DARTS_BF16 ? gemm_workspace_bytes(M, N, K) : 0;
  if (need > workspace_bytes || (need && !d_workspace)) return DARTS_EINVAL;
  hipError_t e = launch_gemm(dtype == DARTS_BF16, d_a, K, d_w, K, d_c, ldc, M, N, K, epilogue,
                             d_workspace, workspace_bytes, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

int darts_debug_gumbel(const float* d_u, float* d_g, int64_t n, void* stream) {
  if ((!d_u || !d_g) && n > 0) return DARTS_EINVAL;
  hipError_t e = launch_gumbel_map(d_u, d_g, n, false, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

int darts_debug_gumbel_fast(const float* d_u, float* d_g, int64_t n, void* stream) {
  if ((!d_u || !d_g) && n > 0) return DARTS_EINVAL;
  hipError_t e = launch_gumbel_map(d_u, d_g, n, true, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

float darts_sampler_gumbel_bound(void) { return gumbel_fast_bound(); }

int darts_group_advantages(const int32_t* d_kept, int32_t n_groups, int32_t k, const float* d_reward,
                           int32_t n_traj, float eps, float* d_adv, void* stream) {
  if (n_groups < 0 || k < 1 || k > 64 || n_traj < 0 || !(eps >= 0.f)) return DARTS_EINVAL;
  if (n_groups > 0 && (!d_kept || !d_reward || !d_adv)) return DARTS_EINVAL;
  hipError_t e = launch_advantages(d_kept, n_groups, k, d_reward, n_traj, eps, d_adv, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

int darts_select_groups(uint8_t* d_status, const int32_t* d_len, const float* d_mean_lp,
                        int32_t n_traj, int32_t m, int32_t k, int32_t L, int32_t m_up,
                        int32_t early_stop, int32_t* d_kept, uint8_t* d_complete,
                        const int32_t* d_page_off, const int32_t* d_pages, int32_t* d_free_out,
                        int32_t* d_n_free, int32_t* d_work, void* stream) {
  if (m < 1 || m > 64 || k < 1 || k > m || n_traj < 0 || n_traj % m) return DARTS_EINVAL;
  if (m < m_up && (L < 1 || L >= k)) return DARTS_EINVAL;
  if (n_traj == 0) return DARTS_OK;
  if (!d_status || !d_len || !d_mean_lp || !d_kept || !d_complete) return DARTS_EINVAL;
  if (d_page_off && (!d_pages || !d_free_out || !d_n_free || !d_work)) return DARTS_EINVAL;
  GroupArgs a{};
  a.status = d_status; a.len = d_len; a.mean_lp = d_mean_lp; a.n_groups = n_traj / m;
  a.m = m; a.k = k; a.L = L; a.m_up = m_up; a.early_stop = early_stop ? 1 : 0;
  a.kept = d_kept; a.complete = d_complete;
  a.page_off = d_page_off; a.pages = d_pages; a.free_out = d_free_out; a.n_free = d_n_free;
  a.work = d_work;
  hipError_t e = launch_select(a, (hipStream_t)stream);
  return e == hipSuccess ? DARTS_OK : DARTS_EHIP;
}

}  // extern "C"
