// Host engine of the DEX library: lattice planner (Algorithm 1's expand /
// insert / validate-and-commit / collapse / advance, Section 3.2), the
// key/value and lattice-slot memory manager, the round executor that drives
// the gfx950 kernels, prefill, and the C ABI declared in include/dex.h.
//
// Device memory layout (all owned by the context):
//   K/V cache     T [L][B][Hkv][E][hd]; entry e < max_context is committed
//                 position e; entries max_context + p*S + i hold lattice slot
//                 i of half p (the two halves alternate at every collapse).
//   slot state    float h [B][2S][d] and sum-of-squares partials
//                 [B][2S][d/16] of each slot's last completed stage, and its
//                 candidate tokens int [B][2S][N].
//   round scratch rows x {h, partials, norm input, q, attention out, SwiGLU
//                 out}, attention split partials, LM-head tile winners; a
//                 stage works in its own row range, so stages may overlap.
// One host->device copy of the round's row tables, one device->host copy of
// the decoded candidates and commits per round.
#include <algorithm>
#include <array>
#include <chrono>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <atomic>
#include <condition_variable>
#include <functional>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "dex.h"
#include "dex_kernels.h"

using namespace dex;

namespace {

// streams a round's stages are spread over unless the caller says otherwise:
// launched per stage, four; grouped, three where a layer's weights take long
// enough to stream that another lane's latency-bound attention and combine
// hide behind them, else one (models whose kernels are bound by launch costs
// gain most from the fewest launches: measured on the 32-layer d4096 and the
// 12-layer d768 models)
constexpr int kDefaultStageStreams = 4;
constexpr int kDefaultGroupedStreams = 3;
constexpr double kLaneLayerBytes = 64e6;

// round phases reported by dex_debug_round_times
constexpr int kRoundPhases = 7;

thread_local std::string g_create_error;

struct Slot {
  int x = 0, pos = 0, parent = -1, fork_stage = -1, c = 0;
  std::vector<int> u;        // candidates of completed stages
  std::vector<int> child;    // child slot per fork stage, -1 if none
};

struct Seq {
  std::vector<int> committed;   // prompt + generated tokens
  std::vector<Slot> slots;      // canonical order, slots[0] = anchor
  int half = 0;                 // lattice half holding the slots
  bool active = false;
  std::vector<int> last_map;
  int last_fresh = -1, last_committed_pos = -1;
};

// Width-cap priority of a work item.  The lattice is a binary tree rooted at
// the anchor's stage-0 node: a depth step (0) goes from a slot's stage k to
// stage k+1, a position step (1) from a slot's stage f to the stage-0 node of
// the slot forked there.  `steps` leads from the root to the node the item
// evaluates; `cost` is the hypothesis cost, sum(f + 1) over the fork stages
// on the way (the length of the path up to its last position step).
struct Item {
  int kind;                 // 0 advance, 1 fork
  int slot, f;
  std::vector<unsigned char> steps;
  int cost;
};

struct Timing {
  int cls;
  hipEvent_t a, b;
  double bytes;
};

// (hypothesis cost, path length, path with the depth step first): path
// length then lexicographic order is the paper's node numbering (depth child
// 2i+1, position child 2i+2) relative to the current anchor.
inline bool item_less(const Item &a, const Item &b) {
  if (a.cost != b.cost) return a.cost < b.cost;
  if (a.steps.size() != b.steps.size()) return a.steps.size() < b.steps.size();
  return a.steps < b.steps;
}

// What the planner needs to know of a context.
struct PlanRule {
  int N, W, decs, max_ctx;
};

}  // namespace

struct dex_ctx {
  // model
  int L, d, H, Hkv, hd, F, V, dtype, es;
  float theta, eps, rscale;
  const void *embed, *lm_head;
  const float *final_norm;
  std::vector<const void *> lw;   // [L][9]
  // config
  std::vector<int> X;
  int N, W, decs, B, max_ctx;
  float temperature = 0.f;               // > 0: sampling mode
  unsigned long long sample_seed = 0;
  hipStream_t stream;
  // stage lanes: lane 0 is `stream`, the others library-owned streams (using
  // the caller's stream as a lane measured ~10 % faster than four library
  // streams: fewer streams than the process's hardware queues to share)
  int n_lanes = 1;
  // grouped launches: the stages of a lane run in step, one launch per
  // kernel and layer step for all of them
  bool grouped = false;
  std::vector<hipStream_t> lane_st;
  std::vector<hipEvent_t> lane_ev;
  hipEvent_t fork_ev = nullptr;
  // lane workers: lanes 1.. enqueue their stages from host threads of their
  // own while the calling thread enqueues lane 0's
  int device = 0;
  std::vector<std::thread> lane_threads;
  std::atomic<int64_t> lane_ticket{0};           // round handed to the workers
  std::atomic<bool> lane_stop{false};
  std::unique_ptr<std::atomic<int64_t>[]> lane_done;  // per lane: last round enqueued
  std::vector<dex_status> lane_status;
  std::vector<std::string> lane_err;
  std::function<dex_status(int)> lane_fn;        // the round's work of a lane
  std::mutex lane_mu;
  std::condition_variable lane_cv;
  std::vector<std::vector<int>> stage_layers;
  // capacities
  int S, R_max, CH_MAX, E, n_part, jmax;
  // packed weights (library-owned, see PackArgs)
  std::vector<void *> p_qkv, p_o, p_gu, p_down;
  void *p_lm = nullptr;
  int ns_d = 0, ns_hhd = 0, ns_F = 0;
  // inducing adapters of the non-final depths: packed W1 [m][d] and W2 [d][m]
  // (library-owned), borrowed norm gains and biases, the gates on the host
  int ad_m = 0, ns_m = 0;
  std::vector<void *> p_ad1, p_ad2;
  std::vector<const float *> ad_norm, ad_b1, ad_b2;
  std::vector<float> ad_alpha;
  void *ad_act = nullptr;                 // [R][m] (T)
  // device buffers
  void *kc = nullptr, *vc = nullptr;
  float2 *rope = nullptr;
  float *bnd_h = nullptr, *bnd_part = nullptr;
  int *cand = nullptr;
  float *h_w = nullptr, *part_w = nullptr, *q_w = nullptr, *attn_part = nullptr;
  void *xb_w = nullptr, *att_w = nullptr, *act_w = nullptr;
  float *ex_h = nullptr, *ex_part = nullptr;
  void *ex_xb = nullptr;
  float2 *amax = nullptr;
  int *u_dev = nullptr;          // [R] decoded candidates, then [2 * commits] (token, k*)
  int *tab_dev = nullptr;
  size_t tab_cap = 0;
  int *job_dev = nullptr;
  // pinned host staging
  int *tab_host = nullptr, *res_host = nullptr, *job_host = nullptr;
  // state
  std::vector<Seq> seqs;
  bool prefilled = false;
  std::atomic<bool> poisoned{false};   // also set by lane workers
  int64_t rounds = 0;
  std::string err;
  float *logits_tap = nullptr;
  int logits_cap = 0;
  // timing
  bool timing = false;
  std::vector<hipEvent_t> ev_pool;
  size_t ev_next = 0;
  std::vector<Timing> pending;
  double t_ms[8] = {0}, t_bytes[8] = {0};
  int64_t t_n[8] = {0};
  // round phases: events on the decode stream at the round's boundaries
  // (two sets, the previous round's last event opens the gap before this one)
  bool round_timing = false;
  hipEvent_t rt_ev[2][6] = {};
  int rt_cur = 0;
  bool rt_prev = false;
  double rt_ms[kRoundPhases] = {0};
  int64_t rt_rounds = 0;
  std::vector<void *> allocs;
};

namespace {

// A failed HIP call leaves device work of the call half done: the context
// is poisoned.
// A lane worker's failures go to its own message (merged by the round).
thread_local std::string *t_lane_err = nullptr;
void hip_failed(dex_ctx *ctx, const char *expr, hipError_t e) {
  const std::string msg = std::string(expr) + ": " + hipGetErrorString(e);
  if (t_lane_err != nullptr) *t_lane_err = msg;
  else ctx->err = msg;
  ctx->poisoned = true;
}
#define HIPCHK(expr)                                                          \
  do {                                                                        \
    hipError_t e_ = (expr);                                                   \
    if (e_ != hipSuccess) {                                                   \
      hip_failed(ctx, #expr, e_);                                             \
      return DEX_E_HIP;                                                       \
    }                                                                         \
  } while (0)

dex_status dalloc(dex_ctx *ctx, void **p, size_t bytes) {
  if (bytes == 0) bytes = 16;
  hipError_t e = hipMalloc(p, bytes);
  if (e != hipSuccess) {
    ctx->err = "hipMalloc of " + std::to_string(bytes) + " bytes failed: " + hipGetErrorString(e);
    *p = nullptr;
    return DEX_E_NOMEM;
  }
  ctx->allocs.push_back(*p);
  return DEX_OK;
}

void dfree(dex_ctx *ctx, void *p) {
  if (!p) return;
  auto it = std::find(ctx->allocs.begin(), ctx->allocs.end(), p);
  if (it != ctx->allocs.end()) ctx->allocs.erase(it);
  (void)hipFree(p);
}

const void *LW(const dex_ctx *ctx, int l, int p) { return ctx->lw[(size_t)l * DEX_P_COUNT + p]; }

// --------------------------------------------------------------- timing
hipEvent_t next_event(dex_ctx *ctx) {
  if (ctx->ev_next >= ctx->ev_pool.size()) {
    hipEvent_t e;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    ctx->ev_pool.push_back(e);
  }
  return ctx->ev_pool[ctx->ev_next++];
}

struct TimedLaunch {
  dex_ctx *ctx;
  int cls;
  double bytes;
  hipEvent_t a = nullptr;
  TimedLaunch(dex_ctx *c, int cl, double b) : ctx(c), cls(cl), bytes(b) {
    if (ctx->timing) {
      a = next_event(ctx);
      if (a) (void)hipEventRecord(a, ctx->stream);
    }
  }
  ~TimedLaunch() {
    if (ctx->timing && a) {
      hipEvent_t b = next_event(ctx);
      if (b) {
        (void)hipEventRecord(b, ctx->stream);
        ctx->pending.push_back({cls, a, b, bytes});
      }
    }
  }
};

void harvest_timing(dex_ctx *ctx) {
  for (auto &t : ctx->pending) {
    float ms = 0.f;
    if (hipEventElapsedTime(&ms, t.a, t.b) == hipSuccess) {
      ctx->t_ms[t.cls] += ms;
      ctx->t_n[t.cls] += 1;
      ctx->t_bytes[t.cls] += t.bytes;
    }
  }
  ctx->pending.clear();
  ctx->ev_next = 0;
}

// ---------------------------------------------------------- lattice rules
std::vector<int> slot_path(const Seq &s, int i) {
  std::vector<int> p;
  while (s.slots[i].parent >= 0) {
    p.push_back(s.slots[i].fork_stage);
    i = s.slots[i].parent;
  }
  std::reverse(p.begin(), p.end());
  return p;
}

std::vector<int> ancestors(const Seq &s, int i) {   // anchor first, parent last
  std::vector<int> a;
  int p = s.slots[i].parent;
  while (p >= 0) {
    a.push_back(p);
    p = s.slots[p].parent;
  }
  std::reverse(a.begin(), a.end());
  return a;
}

// Work items of one round in priority order (anchor first).  Same rule as
// the lattice definition: advance a non-anchor slot only when every ancestor
// completed more stages at round start; fork every completed stage f <= N-2
// not yet forked (without DECS, not when its token repeats a shallower fork
// of the same slot); width cap keeps the anchor and the W-1 items of lowest
// (hypothesis cost, path length, path) -- item_less.
std::vector<Item> plan_items(const PlanRule &rule, const Seq &s) {
  std::vector<Item> items;
  const int N = rule.N;
  for (int i = 0; i < (int)s.slots.size(); ++i) {
    const Slot &sl = s.slots[i];
    std::vector<unsigned char> root;          // steps to this slot's stage-0 node
    int cost = 0;
    for (int f : slot_path(s, i)) {
      root.insert(root.end(), (size_t)f, (unsigned char)0);
      root.push_back(1);
      cost += f + 1;
    }
    bool adv = (i == 0);
    if (!adv) {
      adv = true;
      for (int a : ancestors(s, i))
        if (s.slots[a].c <= sl.c) { adv = false; break; }
    }
    if (adv) {
      std::vector<unsigned char> st = root;
      st.insert(st.end(), (size_t)sl.c, (unsigned char)0);
      items.push_back({0, i, -1, st, cost});
    }
    if (sl.pos + 1 > rule.max_ctx - 1) continue;
    for (int f = 0; f < std::min(sl.c, N - 1); ++f) {
      if (sl.child[f] >= 0) continue;
      if (!rule.decs) {
        bool dup = false;
        for (int g = 0; g < f; ++g) dup |= (sl.u[g] == sl.u[f]);
        if (dup) continue;
      }
      std::vector<unsigned char> st = root;
      st.insert(st.end(), (size_t)f, (unsigned char)0);
      st.push_back(1);
      items.push_back({1, i, f, st, cost + f + 1});
    }
  }
  std::vector<Item> rest(items.begin() + 1, items.end());
  std::sort(rest.begin(), rest.end(), item_less);
  if (rule.W > 0 && (int)rest.size() > rule.W - 1) rest.resize(rule.W - 1);
  std::vector<Item> out;
  out.push_back(items[0]);
  out.insert(out.end(), rest.begin(), rest.end());
  return out;
}

struct Row {
  int seq, slot, stage;
};

inline int slot_entry(const dex_ctx *ctx, const Seq &s, int slot) { return ctx->max_ctx + s.half * ctx->S + slot; }
inline int slot_global(const dex_ctx *ctx, int seq, const Seq &s, int slot) {
  return seq * 2 * ctx->S + s.half * ctx->S + slot;
}

// ------------------------------------------------------- kernel drivers
struct StageTables {
  const int *seq, *pos, *entry, *bnd, *tok, *nc, *chain_off, *chain, *mask_n, *mask_tok, *cand_idx;
  const int *g_row0, *g_nrows, *g_seq, *g_nc;
  int n_groups;
  int n_splits;         // 64-key splits up to the stage's deepest row
  double attn_bytes;    // keys/values a layer's attention reads (algorithmic)
};

double wbytes(const dex_ctx *ctx, double elems) { return elems * ctx->es; }

dex_status run_layers(dex_ctx *ctx, hipStream_t st, int first_layer, int last_layer, int M, const StageTables &t,
                      float *h, float *part, void *xb, float *q, void *att, void *act, float *apart,
                      int jmax, bool to_boundary, const int *bnd_rows) {
  const int d = ctx->d, H = ctx->H, Hkv = ctx->Hkv, hd = ctx->hd, F = ctx->F;
  const size_t layer_kv = (size_t)ctx->B * Hkv * ctx->E * hd * ctx->es;
  for (int l = first_layer; l <= last_layer; ++l) {
    const float alpha = ctx->rscale * (float)(l + 1) / (float)ctx->L;
    // QKV
    {
      GemmArgs a{};
      a.wp = ctx->p_qkv[l]; a.nsteps_w = ctx->ns_d;
      a.N = (H + 2 * Hkv) * hd; a.K = d;
      a.x = xb; a.ldx = d; a.M = M;
      a.part = part; a.n_part = ctx->n_part; a.inv_d = 1.0f / d; a.eps = ctx->eps;
      a.out = q; a.ld_out = H * hd;
      a.kc = (char *)ctx->kc + l * layer_kv; a.vc = (char *)ctx->vc + l * layer_kv;
      a.kv_entries = ctx->E; a.n_heads = H; a.n_kv_heads = Hkv; a.head_dim = hd;
      a.row_seq = t.seq; a.row_pos = t.pos; a.row_entry = t.entry; a.rope = ctx->rope;
      TimedLaunch tl(ctx, 0, wbytes(ctx, (double)a.N * d + (double)M * d + 2.0 * M * Hkv * hd) + 4.0 * M * H * hd);
      HIPCHK(launch_gemm(ctx->dtype, EPI_QKV, a, 1, st));
    }
    // attention + combine
    {
      AttnArgs a{};
      a.q = q; a.ldq = H * hd;
      a.kc = (char *)ctx->kc + l * layer_kv; a.vc = (char *)ctx->vc + l * layer_kv;
      a.kv_entries = ctx->E; a.n_kv_heads = Hkv; a.n_heads = H; a.head_dim = hd; a.batch = ctx->B;
      a.grp_row0 = t.g_row0; a.grp_nrows = t.g_nrows; a.grp_seq = t.g_seq; a.grp_nc = t.g_nc;
      a.row_pos = t.pos; a.row_nc = t.nc; a.row_chain_off = t.chain_off; a.chain = t.chain;
      a.row_seq = t.seq; a.n_rows = M;
      a.part = apart; a.stat = split_stats(apart, M, H, jmax, hd);
      a.jmax = jmax; a.n_splits = t.n_splits; a.scale = 1.0f / std::sqrt((float)hd);
      TimedLaunch tl(ctx, 1, t.attn_bytes);
      HIPCHK(launch_attention(ctx->dtype, a, t.n_groups, st));
    }
    {
      CombineArgs c{};
      c.part = apart; c.stat = split_stats(apart, M, H, jmax, hd);
      c.row_pos = t.pos; c.jmax = jmax; c.n_heads = H; c.head_dim = hd;
      c.out = att; c.ld_out = H * hd;
      TimedLaunch tl(ctx, 2, 0.0);
      HIPCHK(launch_combine(ctx->dtype, c, M, st));
    }
    // O projection + residual
    {
      GemmArgs a{};
      a.wp = ctx->p_o[l]; a.nsteps_w = ctx->ns_hhd; a.N = d; a.K = H * hd;
      a.x = att; a.ldx = H * hd; a.M = M;
      a.h = h; a.ld_h = d; a.alpha = alpha;
      a.g_next = (const float *)LW(ctx, l, DEX_P_FFN_NORM); a.xb = xb;
      a.part_out = part; a.n_part_out = ctx->n_part;
      TimedLaunch tl(ctx, 3, wbytes(ctx, (double)d * H * hd + (double)M * H * hd + (double)M * d) + 8.0 * M * d);
      HIPCHK(launch_gemm(ctx->dtype, EPI_RESID, a, 1, st));
    }
    // gate/up + SiLU
    {
      GemmArgs a{};
      a.wp = ctx->p_gu[l]; a.nsteps_w = ctx->ns_d;
      a.N = F; a.K = d;
      a.x = xb; a.ldx = d; a.M = M;
      a.part = part; a.n_part = ctx->n_part; a.inv_d = 1.0f / d; a.eps = ctx->eps;
      a.act = act; a.ld_act = F;
      TimedLaunch tl(ctx, 4, wbytes(ctx, 2.0 * F * d + (double)M * d + (double)M * F));
      HIPCHK(launch_gemm(ctx->dtype, EPI_SWIGLU, a, 1, st));
    }
    // down + residual
    {
      const bool last = (l == last_layer);
      GemmArgs a{};
      a.wp = ctx->p_down[l]; a.nsteps_w = ctx->ns_F; a.N = d; a.K = F;
      a.x = act; a.ldx = F; a.M = M;
      a.h = h; a.ld_h = d; a.alpha = alpha;
      a.g_next = last ? nullptr : (const float *)LW(ctx, l + 1, DEX_P_ATTN_NORM);
      a.xb = last ? nullptr : xb;
      a.part_out = part; a.n_part_out = ctx->n_part;
      if (last && to_boundary) {
        a.row_bnd = bnd_rows; a.bnd_h = ctx->bnd_h; a.bnd_part = ctx->bnd_part;
      }
      TimedLaunch tl(ctx, 5, wbytes(ctx, (double)d * F + (double)M * F + (double)M * d) + 8.0 * M * d);
      HIPCHK(launch_gemm(ctx->dtype, EPI_RESID, a, 1, st));
    }
  }
  return DEX_OK;
}

// Rows [r0, r0 + M) of the exit buffers from their source states, with the
// next norm's input g * h.
dex_status exit_prep(dex_ctx *ctx, int r0, int M, const int *row_src, const float *src_h, const float *src_part,
                     const float *g) {
  if (M <= 0) return DEX_OK;
  PrepArgs p{};
  p.M = M; p.d = ctx->d; p.n_part = ctx->n_part; p.embed_rows = 0;
  p.row_src = row_src + r0; p.bnd_h = src_h; p.bnd_part = src_part; p.g = g;
  p.h = ctx->ex_h + (size_t)r0 * ctx->d; p.part = ctx->ex_part + (size_t)r0 * ctx->n_part;
  p.xb = (char *)ctx->ex_xb + (size_t)r0 * ctx->d * ctx->es;
  TimedLaunch tl(ctx, 7, 0.0);
  HIPCHK(launch_prep(ctx->dtype, p, ctx->stream));
  return DEX_OK;
}

// Inducing adapter of non-final depth k on exit rows [r0, r0 + M), whose
// states and g_k * h are in the exit buffers: h <- h + alpha (W2 silu(W1
// RMSNorm(h; g_k) + b1) + b2), then the final norm's input and partials.
dex_status exit_adapter(dex_ctx *ctx, int k, int r0, int M) {
  if (M <= 0) return DEX_OK;
  const int d = ctx->d, m = ctx->ad_m;
  void *xb = (char *)ctx->ex_xb + (size_t)r0 * d * ctx->es;
  float *part = ctx->ex_part + (size_t)r0 * ctx->n_part;
  void *act = (char *)ctx->ad_act + (size_t)r0 * m * ctx->es;
  {
    GemmArgs a{};
    a.wp = ctx->p_ad1[k]; a.nsteps_w = ctx->ns_d; a.N = m; a.K = d;
    a.x = xb; a.ldx = d; a.M = M; a.part = part; a.n_part = ctx->n_part; a.inv_d = 1.0f / d; a.eps = ctx->eps;
    a.act = act; a.ld_act = m; a.bias = ctx->ad_b1[k];
    TimedLaunch tl(ctx, 7, 0.0);
    HIPCHK(launch_gemm(ctx->dtype, EPI_BIAS_SILU, a, 1, ctx->stream));
  }
  {
    GemmArgs a{};
    a.wp = ctx->p_ad2[k]; a.nsteps_w = ctx->ns_m; a.N = d; a.K = m;
    a.x = act; a.ldx = m; a.M = M;
    a.h = ctx->ex_h + (size_t)r0 * d; a.ld_h = d; a.alpha = ctx->ad_alpha[k]; a.bias = ctx->ad_b2[k];
    a.g_next = ctx->final_norm; a.xb = xb; a.part_out = part; a.n_part_out = ctx->n_part;
    TimedLaunch tl(ctx, 7, 0.0);
    HIPCHK(launch_gemm(ctx->dtype, EPI_RESID, a, 1, ctx->stream));
  }
  return DEX_OK;
}

// exit head over M rows whose final state sits in (src_h, src_part)[row_src[m]];
// stage_r0 (host, N + 1 bounds of the stage-major rows) selects the rows of
// non-final depths for the adapters (nullptr: every row is final depth)
dex_status run_exit(dex_ctx *ctx, int M, const int *row_src, const float *src_h, const float *src_part,
                    const int *mask_n, const int *mask_tok, const int *cand_idx, int *cand, const int *row_seq,
                    const int *row_pos, const int *stage_r0, const int *row_commit) {
  const hipStream_t st = ctx->stream;
  if (ctx->ad_m > 0 && stage_r0 != nullptr) {
    const int N = ctx->N;
    for (int k = 0; k + 1 < N; ++k) {
      const int b0 = stage_r0[k], nb = stage_r0[k + 1] - b0;
      dex_status s1 = exit_prep(ctx, b0, nb, row_src, src_h, src_part, ctx->ad_norm[k]);
      if (s1 == DEX_OK) s1 = exit_adapter(ctx, k, b0, nb);
      if (s1 != DEX_OK) return s1;
    }
    dex_status s2 = exit_prep(ctx, stage_r0[N - 1], M - stage_r0[N - 1], row_src, src_h, src_part, ctx->final_norm);
    if (s2 != DEX_OK) return s2;
  } else {
    dex_status s2 = exit_prep(ctx, 0, M, row_src, src_h, src_part, ctx->final_norm);
    if (s2 != DEX_OK) return s2;
  }
  const int n_tiles = (ctx->V + 15) / 16;
  {
    GemmArgs a{};
    a.wp = ctx->p_lm; a.nsteps_w = ctx->ns_d; a.N = ctx->V; a.K = ctx->d;
    a.x = ctx->ex_xb; a.ldx = ctx->d; a.M = M;
    a.part = ctx->ex_part; a.n_part = ctx->n_part; a.inv_d = 1.0f / ctx->d; a.eps = ctx->eps;
    a.mask_n = mask_n; a.mask_tok = mask_tok; a.mask_stride = ctx->N;
    a.logits_tap = ctx->logits_tap; a.amax = ctx->amax; a.n_tiles = n_tiles;
    a.temperature = ctx->temperature; a.sample_seed = ctx->sample_seed; a.row_seq = row_seq; a.row_pos = row_pos;
    TimedLaunch tl(ctx, 6, wbytes(ctx, (double)ctx->V * ctx->d + (double)M * ctx->d));
    HIPCHK(launch_gemm(ctx->dtype, EPI_LOGITS, a, 1, st));
  }
  {
    ArgmaxArgs g{};
    g.amax = ctx->amax; g.n_tiles = n_tiles; g.M = M; g.u_out = ctx->u_dev;
    g.cand = cand; g.row_cand = cand_idx;
    g.row_commit = row_commit; g.N = ctx->N; g.commit_out = ctx->u_dev + M;
    TimedLaunch tl(ctx, 7, 0.0);
    HIPCHK(launch_argmax(g, st));
  }
  return DEX_OK;
}

// Argument errors and a full context leave the state as it was; any other
// failure poisons it.
dex_status fail(dex_ctx *ctx, dex_status s) {
  if (s != DEX_OK && s != DEX_E_INVAL && s != DEX_E_CAPACITY) ctx->poisoned = true;
  return s;
}

// A failure after the round's planning has changed the lattice.
dex_status fail_mid_round(dex_ctx *ctx, const char *msg, dex_status s) {
  ctx->err = msg;
  ctx->poisoned = true;
  return s;
}

// ------------------------------------------------ stand-alone attention
// One call of the stand-alone decode attention (the arguments of
// dex_debug_attention).
struct AttnCall {
  int dtype, head_dim, n_heads, n_kv_heads, batch, kv_entries;
  const void *k_cache, *v_cache;
  const float *q;
  int n_rows;
  const int32_t *row_seq, *row_pos, *row_nc, *chain_off, *chain;
  int chain_len;
  void *out;
};

// Offsets (in ints) of the device row tables, the row-group count, the split
// count and the split partials' size of one call.
struct AttnTab {
  size_t o_pos, o_nc, o_seq, o_coff, o_g0, o_gn, o_gs, o_gc, o_chain, n_ints;
  int ng, n_splits;
  size_t part_bytes;
};

size_t attention_table_ints(int n_rows, int chain_len) { return 8 * (size_t)n_rows + (size_t)chain_len + 1; }

// Validates a call on the host (nothing is launched for a bad one) and
// writes its row tables to tab (cap ints, at least attention_table_ints):
// row groups are consecutive rows of one sequence sharing their committed
// prefix, at most 64 (row, query head) pairs' worth of rows each.
dex_status attention_tables(const AttnCall &c, int *tab, size_t cap, AttnTab *t) {
  if (c.dtype != DEX_F32 && c.dtype != DEX_BF16) return DEX_E_INVAL;
  if (c.head_dim != 32 && c.head_dim != 64 && c.head_dim != 128) return DEX_E_INVAL;
  if (c.n_kv_heads < 1 || c.n_heads < c.n_kv_heads || c.n_heads % c.n_kv_heads || c.n_heads / c.n_kv_heads > 8)
    return DEX_E_INVAL;
  if (c.batch < 1 || c.kv_entries < 1 || c.n_rows < 1 || c.chain_len < 0) return DEX_E_INVAL;
  if (!c.k_cache || !c.v_cache || !c.q || !c.out || !c.row_seq || !c.row_pos || !c.row_nc || !c.chain_off)
    return DEX_E_INVAL;
  if (c.chain_len > 0 && !c.chain) return DEX_E_INVAL;
  if (cap < attention_table_ints(c.n_rows, c.chain_len)) return DEX_E_INVAL;
  int maxpos = 0;
  for (int r = 0; r < c.n_rows; ++r) {
    const int sq = c.row_seq[r], pos = c.row_pos[r], nc = c.row_nc[r], co = c.chain_off[r];
    if (sq < 0 || sq >= c.batch || pos < 0 || pos >= c.kv_entries || nc < 0 || nc > pos + 1) return DEX_E_INVAL;
    if (pos - nc >= ATT_SPLIT) return DEX_E_INVAL;
    if (nc <= pos && (co < 0 || (int64_t)co + (pos - nc) >= c.chain_len)) return DEX_E_INVAL;
    for (int i = 0; nc + i <= pos; ++i)
      if (c.chain[co + i] < 0 || c.chain[co + i] >= c.kv_entries) return DEX_E_INVAL;
    maxpos = std::max(maxpos, pos);
  }
  t->n_splits = maxpos / ATT_SPLIT + 1;
  if (t->n_splits > ATT_MAX_SPLITS) return DEX_E_INVAL;
  const int R = c.n_rows;
  t->o_pos = 0; t->o_nc = R; t->o_seq = 2 * (size_t)R; t->o_coff = 3 * (size_t)R; t->o_g0 = 4 * (size_t)R;
  std::copy(c.row_pos, c.row_pos + R, tab + t->o_pos);
  std::copy(c.row_nc, c.row_nc + R, tab + t->o_nc);
  std::copy(c.row_seq, c.row_seq + R, tab + t->o_seq);
  std::copy(c.chain_off, c.chain_off + R, tab + t->o_coff);
  const int G = c.n_heads / c.n_kv_heads, grp_rows = std::max(1, ATT_MAX_PAIRS / G);
  int ng = 0;
  int *g0 = tab + t->o_g0;
  for (int r = 0; r < R;) {                 // group starts; sizes and sequences below
    int e = r;
    while (e < R && c.row_seq[e] == c.row_seq[r] && c.row_nc[e] == c.row_nc[r] && e - r < grp_rows) ++e;
    g0[ng++] = r;
    r = e;
  }
  t->ng = ng;
  t->o_gn = t->o_g0 + ng; t->o_gs = t->o_gn + ng; t->o_gc = t->o_gs + ng; t->o_chain = t->o_gc + ng;
  for (int g = 0; g < ng; ++g) {
    const int e = g + 1 < ng ? g0[g + 1] : R;
    tab[t->o_gn + g] = e - g0[g];
    tab[t->o_gs + g] = c.row_seq[g0[g]];
    tab[t->o_gc + g] = c.row_nc[g0[g]];
  }
  if (c.chain_len > 0) std::copy(c.chain, c.chain + c.chain_len, tab + t->o_chain);
  else tab[t->o_chain] = 0;
  t->n_ints = t->o_chain + std::max(c.chain_len, 1);
  t->part_bytes = (size_t)R * c.n_heads * t->n_splits * (c.head_dim + 2) * 4;
  return DEX_OK;
}

// The decode attention and its split combine over device tables dtab (laid
// out by attention_tables) with split partials in part.
hipError_t launch_attention_call(const AttnCall &c, const AttnTab &t, const int *dtab, float *part,
                                 hipStream_t st) {
  AttnArgs a{};
  a.q = c.q; a.ldq = c.n_heads * c.head_dim; a.kc = c.k_cache; a.vc = c.v_cache; a.kv_entries = c.kv_entries;
  a.n_kv_heads = c.n_kv_heads; a.n_heads = c.n_heads; a.head_dim = c.head_dim; a.batch = c.batch;
  a.grp_row0 = dtab + t.o_g0; a.grp_nrows = dtab + t.o_gn; a.grp_seq = dtab + t.o_gs; a.grp_nc = dtab + t.o_gc;
  a.row_pos = dtab + t.o_pos; a.row_nc = dtab + t.o_nc; a.row_chain_off = dtab + t.o_coff;
  a.chain = dtab + t.o_chain; a.row_seq = dtab + t.o_seq; a.n_rows = c.n_rows; a.part = part;
  a.stat = split_stats(part, c.n_rows, c.n_heads, t.n_splits, c.head_dim);
  a.jmax = t.n_splits; a.n_splits = t.n_splits; a.scale = 1.0f / std::sqrt((float)c.head_dim);
  hipError_t e = launch_attention(c.dtype, a, t.ng, st);
  CombineArgs cb{};
  cb.part = part; cb.stat = a.stat; cb.row_pos = dtab + t.o_pos; cb.jmax = t.n_splits; cb.n_heads = c.n_heads;
  cb.head_dim = c.head_dim; cb.out = c.out; cb.ld_out = c.n_heads * c.head_dim;
  if (e == hipSuccess) e = launch_combine(c.dtype, cb, c.n_rows, st);
  return e;
}

// ------------------------------------------ fixed scratch (no allocation)
// dex_debug_attention_noalloc keeps its row tables and split partials in
// this array instead of allocating them.  Host code never uses the array's
// name as a device address: scratch_address() resolves it once per device
// (with that device current) and every kernel argument, copy or fill uses
// the resolved address.
constexpr size_t kScratchBytes = 64ull << 20;
constexpr size_t kScratchTableBytes = 256ull << 10;
constexpr int kNoallocMaxChain = 16384;
constexpr size_t kNoallocTableInts = 8 * DEX_MAX_ROWS + kNoallocMaxChain + 1;
static_assert(kNoallocTableInts * 4 <= kScratchTableBytes, "row tables fit their scratch region");

static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_addr[kMaxDevices] = {};

hipError_t scratch_address(void **out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (g_scratch_addr[dev] == nullptr) {
    void *p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_scratch_addr[dev] = p;
  }
  *out = g_scratch_addr[dev];
  return hipSuccess;
}

// A lane worker: waits for a round (spinning for half a millisecond, then
// sleeping in 2 ms slices), enqueues its lane's stages, reports.
void lane_worker(dex_ctx *ctx, int lane) {
  (void)hipSetDevice(ctx->device);
  int64_t seen = 0;
  for (;;) {
    const auto t0 = std::chrono::steady_clock::now();
    int64_t t;
    while ((t = ctx->lane_ticket.load(std::memory_order_acquire)) == seen) {
      if (ctx->lane_stop.load(std::memory_order_acquire)) return;
      if (std::chrono::steady_clock::now() - t0 < std::chrono::microseconds(500)) continue;
      std::unique_lock<std::mutex> lk(ctx->lane_mu);
      ctx->lane_cv.wait_for(lk, std::chrono::milliseconds(2), [&] {
        return ctx->lane_ticket.load(std::memory_order_acquire) != seen ||
               ctx->lane_stop.load(std::memory_order_acquire);
      });
    }
    seen = t;
    std::string err;
    t_lane_err = &err;
    const dex_status st = ctx->lane_fn(lane);
    t_lane_err = nullptr;
    ctx->lane_status[lane] = st;
    ctx->lane_err[lane] = std::move(err);
    ctx->lane_done[lane].store(t, std::memory_order_release);
  }
}

void stop_lane_workers(dex_ctx *ctx) {
  if (ctx->lane_threads.empty()) return;
  {
    std::lock_guard<std::mutex> lk(ctx->lane_mu);
    ctx->lane_stop.store(true, std::memory_order_release);
  }
  ctx->lane_cv.notify_all();
  for (auto &th : ctx->lane_threads) th.join();
  ctx->lane_threads.clear();
}

}  // namespace

// ===================================================================== ABI
extern "C" {

const char *dex_last_error(const dex_ctx *ctx) {
  if (ctx == nullptr) return g_create_error.c_str();
  return ctx->err.c_str();
}

void dex_destroy(dex_ctx *ctx) {
  if (!ctx) return;
  stop_lane_workers(ctx);
  if (ctx->stream) (void)hipStreamSynchronize(ctx->stream);
  else (void)hipDeviceSynchronize();
  for (void *p : ctx->allocs) (void)hipFree(p);
  if (ctx->tab_host) (void)hipHostFree(ctx->tab_host);
  if (ctx->res_host) (void)hipHostFree(ctx->res_host);
  if (ctx->job_host) (void)hipHostFree(ctx->job_host);
  for (auto e : ctx->ev_pool) (void)hipEventDestroy(e);
  for (size_t i = 0; i < ctx->lane_st.size(); ++i) {
    if (!ctx->lane_st[i] || ctx->lane_st[i] == ctx->stream) continue;
    (void)hipStreamSynchronize(ctx->lane_st[i]);
    (void)hipStreamDestroy(ctx->lane_st[i]);
  }
  for (auto e : ctx->lane_ev) if (e) (void)hipEventDestroy(e);
  for (auto &set : ctx->rt_ev)
    for (auto e : set) if (e) (void)hipEventDestroy(e);
  if (ctx->fork_ev) (void)hipEventDestroy(ctx->fork_ev);
  delete ctx;
}

dex_status dex_create(const dex_model *m, const dex_config *c, dex_ctx **out) {
  g_create_error.clear();
  if (!out) { g_create_error = "out is NULL"; return DEX_E_INVAL; }
  *out = nullptr;
  if (!m || !c) { g_create_error = "model or config is NULL"; return DEX_E_INVAL; }
  auto bad = [](const std::string &s) { g_create_error = s; return DEX_E_INVAL; };
  if (m->n_layers < 1 || m->d_model < 16 || m->d_model % 16 || m->n_heads < 1 || m->n_kv_heads < 1 ||
      m->n_heads % m->n_kv_heads || m->head_dim < 16 || m->head_dim % 16 || m->head_dim > 128 ||
      m->d_ffn < 1 || m->vocab < 2)
    return bad("model dimensions out of range");
  if (m->n_heads / m->n_kv_heads > 8) return bad("n_heads / n_kv_heads must be <= 8");
  // the attention kernels exist for these head sizes only
  if (m->head_dim != 32 && m->head_dim != 64 && m->head_dim != 128) return bad("head_dim must be 32, 64 or 128");
  if (m->weight_dtype != DEX_F32 && m->weight_dtype != DEX_BF16) return bad("weight_dtype must be DEX_F32 or DEX_BF16");
  const int epb = m->weight_dtype == DEX_BF16 ? 8 : 4;
  if (m->d_ffn % epb || (m->n_heads * m->head_dim) % epb) return bad("d_ffn must be a multiple of 8 (bf16) / 4 (f32)");
  if (!m->embed || !m->final_norm || !m->lm_head || !m->layers) return bad("null weight pointer");
  for (int i = 0; i < m->n_layers * DEX_P_COUNT; ++i)
    if (!m->layers[i]) return bad("null layer weight pointer");
  if (!(m->rms_eps >= 0.f) || !(m->rope_theta > 0.f)) return bad("rms_eps / rope_theta out of range");
  if (c->n_explored < 1 || c->n_explored > DEX_MAX_EXPLORED || !c->explored) return bad("n_explored out of range");
  for (int i = 0; i < c->n_explored; ++i) {
    const int dd = c->explored[i];
    if (dd < 1 || dd > m->n_layers || (i > 0 && dd <= c->explored[i - 1]))
      return bad("explored depths must be strictly increasing in [1, L]");
  }
  if (c->explored[c->n_explored - 1] != m->n_layers) return bad("the last explored depth must be L");
  if (c->batch < 1 || c->batch > DEX_MAX_BATCH) return bad("batch out of range");
  if (c->width_cap < 0) return bad("width_cap must be >= 0");
  if (c->max_context < 2) return bad("max_context must be >= 2");
  if (!(c->temperature >= 0.f) || !std::isfinite(c->temperature)) return bad("temperature must be finite and >= 0");
  if (c->adapter_dim < 0) return bad("adapter_dim must be >= 0");
  if (c->adapter_dim > 0) {
    if (c->adapter_dim % epb) return bad("adapter_dim must be a multiple of 8 (bf16) / 4 (f32)");
    if (!c->adapters) return bad("adapter_dim > 0 needs the adapter pointers");
    for (int i = 0; i < (c->n_explored - 1) * 6; ++i)
      if (!c->adapters[i]) return bad("null adapter pointer");
  }
  if ((c->max_context + ATT_SPLIT - 1) / ATT_SPLIT > ATT_MAX_SPLITS) return bad("max_context too long");
  const int N = c->n_explored;
  long long per_seq = c->width_cap > 0 ? c->width_cap : (N - 1 >= 20 ? (1LL << 20) : (1LL << (N - 1)));
  if (per_seq * c->batch > DEX_MAX_ROWS) return bad("rows per round exceed DEX_MAX_ROWS (lower width_cap or batch)");

  dex_ctx *ctx = new dex_ctx();
  ctx->L = m->n_layers; ctx->d = m->d_model; ctx->H = m->n_heads; ctx->Hkv = m->n_kv_heads;
  ctx->hd = m->head_dim; ctx->F = m->d_ffn; ctx->V = m->vocab; ctx->dtype = m->weight_dtype;
  ctx->es = ctx->dtype == DEX_BF16 ? 2 : 4;
  ctx->theta = m->rope_theta; ctx->eps = m->rms_eps; ctx->rscale = m->residual_scale;
  ctx->embed = m->embed; ctx->lm_head = m->lm_head; ctx->final_norm = m->final_norm;
  ctx->lw.assign(m->layers, m->layers + (size_t)m->n_layers * DEX_P_COUNT);
  ctx->X.assign(c->explored, c->explored + N);
  ctx->N = N; ctx->W = c->width_cap; ctx->decs = c->decs ? 1 : 0; ctx->B = c->batch;
  ctx->max_ctx = c->max_context; ctx->stream = (hipStream_t)c->hip_stream;
  ctx->temperature = c->temperature; ctx->sample_seed = c->sample_seed;
  int prev = 0;
  for (int k = 0; k < N; ++k) {
    std::vector<int> ls;
    for (int l = prev; l < ctx->X[k]; ++l) ls.push_back(l);
    ctx->stage_layers.push_back(ls);
    prev = ctx->X[k];
  }
  ctx->R_max = (int)per_seq * ctx->B;
  ctx->S = ctx->W > 0 ? N * ctx->W + 1 : (int)per_seq;
  ctx->CH_MAX = N + 1;
  ctx->E = ctx->max_ctx + 2 * ctx->S;
  ctx->n_part = ctx->d / 16;
  ctx->jmax = (ctx->max_ctx + ATT_SPLIT - 1) / ATT_SPLIT;

  dex_status st = DEX_OK;
  auto A = [&](void **p, size_t bytes) {
    if (st == DEX_OK) st = dalloc(ctx, p, bytes);
  };
  const size_t R = ctx->R_max, d = ctx->d, es = ctx->es;
  const size_t kv_bytes = (size_t)ctx->L * ctx->B * ctx->Hkv * ctx->E * ctx->hd * es;
  A(&ctx->kc, kv_bytes);
  A(&ctx->vc, kv_bytes);
  A((void **)&ctx->rope, (size_t)ctx->max_ctx * (ctx->hd / 2) * sizeof(float2));
  const size_t slots_total = (size_t)ctx->B * 2 * ctx->S;
  A((void **)&ctx->bnd_h, slots_total * d * 4);
  A((void **)&ctx->bnd_part, slots_total * ctx->n_part * 4);
  A((void **)&ctx->cand, slots_total * N * 4);
  A((void **)&ctx->h_w, R * d * 4);
  A((void **)&ctx->part_w, R * ctx->n_part * 4);
  A(&ctx->xb_w, R * d * es);
  A((void **)&ctx->q_w, R * ctx->H * ctx->hd * 4);
  A(&ctx->att_w, R * ctx->H * ctx->hd * es);
  A(&ctx->act_w, R * ctx->F * es);
  A((void **)&ctx->attn_part, R * ctx->H * ctx->jmax * (ctx->hd + 2) * 4);
  A((void **)&ctx->ex_h, R * d * 4);
  A((void **)&ctx->ex_part, R * ctx->n_part * 4);
  A(&ctx->ex_xb, R * d * es);
  if (c->adapter_dim > 0) A(&ctx->ad_act, R * (size_t)c->adapter_dim * es);
  A((void **)&ctx->amax, R * ((ctx->V + 15) / 16) * sizeof(float2));
  A((void **)&ctx->u_dev, (R + 2 * (size_t)ctx->B) * 4 + 256);
  A((void **)&ctx->job_dev, (size_t)(ctx->B * (ctx->S + 1)) * 6 * 4 + 256);
  ctx->tab_cap = (size_t)R * (16 + 2 * N + ctx->CH_MAX) + 4 * ctx->B + 1024;
  A((void **)&ctx->tab_dev, ctx->tab_cap * 4);

  if (st != DEX_OK) {
    g_create_error = ctx->err;
    dex_destroy(ctx);
    return st;
  }
  if (hipHostMalloc((void **)&ctx->tab_host, ctx->tab_cap * 4) != hipSuccess ||
      hipHostMalloc((void **)&ctx->res_host, (R + 2 * ctx->B + 64) * 4) != hipSuccess ||
      hipHostMalloc((void **)&ctx->job_host, (size_t)(ctx->B * (ctx->S + 1)) * 6 * 4 + 256) != hipSuccess) {
    g_create_error = "hipHostMalloc failed";
    dex_destroy(ctx);
    return DEX_E_NOMEM;
  }
  // RoPE table in double precision, rounded once: (cos, sin)(p * theta^(-2i/hd))
  {
    std::vector<float2> tab((size_t)ctx->max_ctx * (ctx->hd / 2));
    for (int p = 0; p < ctx->max_ctx; ++p)
      for (int i = 0; i < ctx->hd / 2; ++i) {
        const double ang = (double)p * std::pow((double)ctx->theta, -2.0 * i / (double)ctx->hd);
        tab[(size_t)p * (ctx->hd / 2) + i] = make_float2((float)std::cos(ang), (float)std::sin(ang));
      }
    hipError_t e = hipMemcpy(ctx->rope, tab.data(), tab.size() * sizeof(float2), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipMemset(ctx->kc, 0, kv_bytes);
    if (e == hipSuccess) e = hipMemset(ctx->vc, 0, kv_bytes);
    if (e == hipSuccess) e = hipMemset(ctx->cand, 0xff, slots_total * N * 4);

    if (e != hipSuccess) {
      g_create_error = std::string("initialisation copy failed: ") + hipGetErrorString(e);
      dex_destroy(ctx);
      return DEX_E_HIP;
    }
  }
  // packed weights: every wave load of the skinny GEMMs reads 1 KB contiguously
  {
    const int kstep = ctx->dtype == DEX_BF16 ? 32 : 16;
    ctx->ns_d = (ctx->d + kstep - 1) / kstep;
    ctx->ns_hhd = (ctx->H * ctx->hd + kstep - 1) / kstep;
    ctx->ns_F = (ctx->F + kstep - 1) / kstep;
    const int H = ctx->H, Hkv = ctx->Hkv, hd = ctx->hd, dd = ctx->d, F = ctx->F;
    auto pack = [&](void **dst, const void *w0, const void *w1, const void *w2, int n0, int n1, int n2, int N,
                    int K, int mode) -> dex_status {
      dex_status s2 = dalloc(ctx, dst, packed_bytes(ctx->dtype, N, K, mode));
      if (s2 != DEX_OK) return s2;
      PackArgs pa{};
      pa.w0 = w0; pa.w1 = w1; pa.w2 = w2; pa.n0 = n0; pa.n1 = n1; pa.n2 = n2;
      pa.N = N; pa.K = K; pa.mode = mode; pa.head_dim = hd; pa.out = *dst;
      hipError_t e = launch_pack(ctx->dtype, pa, nullptr);
      if (e != hipSuccess) { ctx->err = std::string("weight packing failed: ") + hipGetErrorString(e); return DEX_E_HIP; }
      return DEX_OK;
    };
    ctx->p_qkv.assign(ctx->L, nullptr); ctx->p_o.assign(ctx->L, nullptr);
    ctx->p_gu.assign(ctx->L, nullptr); ctx->p_down.assign(ctx->L, nullptr);
    dex_status ps = DEX_OK;
    for (int l = 0; l < ctx->L && ps == DEX_OK; ++l) {
      ps = pack(&ctx->p_qkv[l], LW(ctx, l, DEX_P_WQ), LW(ctx, l, DEX_P_WK), LW(ctx, l, DEX_P_WV), H * hd, Hkv * hd,
                Hkv * hd, (H + 2 * Hkv) * hd, dd, 1);
      if (ps == DEX_OK) ps = pack(&ctx->p_o[l], LW(ctx, l, DEX_P_WO), nullptr, nullptr, dd, 0, 0, dd, H * hd, 0);
      if (ps == DEX_OK)
        ps = pack(&ctx->p_gu[l], LW(ctx, l, DEX_P_W_GATE), LW(ctx, l, DEX_P_W_UP), nullptr, F, F, 0, F, dd, 2);
      if (ps == DEX_OK) ps = pack(&ctx->p_down[l], LW(ctx, l, DEX_P_W_DOWN), nullptr, nullptr, dd, 0, 0, dd, F, 0);
    }
    if (ps == DEX_OK) ps = pack(&ctx->p_lm, ctx->lm_head, nullptr, nullptr, ctx->V, 0, 0, ctx->V, dd, 0);
    if (ps == DEX_OK && c->adapter_dim > 0) {
      const int am = c->adapter_dim;
      ctx->ad_m = am;
      ctx->ns_m = (am + kstep - 1) / kstep;
      ctx->p_ad1.assign(N - 1, nullptr); ctx->p_ad2.assign(N - 1, nullptr);
      ctx->ad_norm.assign(N - 1, nullptr); ctx->ad_b1.assign(N - 1, nullptr); ctx->ad_b2.assign(N - 1, nullptr);
      ctx->ad_alpha.assign(N - 1, 0.f);
      for (int k = 0; k + 1 < N && ps == DEX_OK; ++k) {
        const void *const *ap = c->adapters + (size_t)k * 6;
        ctx->ad_norm[k] = (const float *)ap[0];
        ctx->ad_b1[k] = (const float *)ap[2];
        ctx->ad_b2[k] = (const float *)ap[4];
        ps = pack(&ctx->p_ad1[k], ap[1], nullptr, nullptr, am, 0, 0, am, dd, 0);
        if (ps == DEX_OK) ps = pack(&ctx->p_ad2[k], ap[3], nullptr, nullptr, dd, 0, 0, dd, am, 0);
        if (ps == DEX_OK && hipMemcpy(&ctx->ad_alpha[k], ap[5], sizeof(float), hipMemcpyDeviceToHost) != hipSuccess) {
          ctx->err = "reading an adapter gate failed";
          ps = DEX_E_HIP;
        }
      }
    }
    if (ps == DEX_OK && hipDeviceSynchronize() != hipSuccess) { ctx->err = "weight packing failed"; ps = DEX_E_HIP; }
    if (ps != DEX_OK) {
      g_create_error = ctx->err;
      dex_destroy(ctx);
      return ps;
    }
  }
  // stage lanes (default priority, non-blocking streams)
  {
    ctx->grouped = c->stage_grouping >= 0;
    const double layer_bytes = (double)ctx->es * ((double)ctx->d * (ctx->H + 2 * ctx->Hkv) * ctx->hd +
                                                   (double)ctx->H * ctx->hd * ctx->d + 3.0 * ctx->d * ctx->F);
    const int def_lanes = !ctx->grouped ? kDefaultStageStreams
                          : layer_bytes >= kLaneLayerBytes ? kDefaultGroupedStreams : 1;
    ctx->n_lanes = c->stage_streams > 0 ? std::min<int>(c->stage_streams, 8) : def_lanes;
    ctx->lane_st.assign(ctx->n_lanes, ctx->stream);
    ctx->lane_ev.assign(ctx->n_lanes, nullptr);
    hipError_t e = hipSuccess;
    if (ctx->n_lanes > 1) {
      e = hipEventCreateWithFlags(&ctx->fork_ev, hipEventDisableTiming);
      for (int i = 1; i < ctx->n_lanes && e == hipSuccess; ++i) {
        e = hipStreamCreateWithFlags(&ctx->lane_st[i], hipStreamNonBlocking);
        if (e != hipSuccess) { ctx->lane_st[i] = nullptr; break; }
      }
      for (int i = 1; i < ctx->n_lanes && e == hipSuccess; ++i)
        e = hipEventCreateWithFlags(&ctx->lane_ev[i], hipEventDisableTiming);
    }
    if (e != hipSuccess) {
      g_create_error = std::string("stream creation failed: ") + hipGetErrorString(e);
      dex_destroy(ctx);
      return DEX_E_HIP;
    }
    // each extra lane issues its stages from a host thread of its own: the
    // host needs ~2.5 us per launch, which bounds the rounds of models with
    // short kernels, and issuing the lanes one after another also staggers
    // their starts on larger models
    if (ctx->n_lanes > 1) {
      (void)hipGetDevice(&ctx->device);
      ctx->lane_done.reset(new std::atomic<int64_t>[ctx->n_lanes]());
      ctx->lane_status.assign(ctx->n_lanes, DEX_OK);
      ctx->lane_err.assign(ctx->n_lanes, std::string());
      try {
        for (int i = 1; i < ctx->n_lanes; ++i) ctx->lane_threads.emplace_back(lane_worker, ctx, i);
      } catch (...) {
        stop_lane_workers(ctx);       // fewer threads: the calling thread issues every lane
      }
    }
  }
  ctx->seqs.resize(ctx->B);
  *out = ctx;
  return DEX_OK;
}

dex_status dex_prefill(dex_ctx *ctx, const int32_t *prompts, int32_t P, int32_t *first) {
  if (!ctx) return DEX_E_INVAL;
  if (ctx->poisoned) { ctx->err = "context poisoned by an earlier failure"; return DEX_E_STATE; }
  if (!prompts || !first || P < 1) { ctx->err = "bad prefill arguments"; return DEX_E_INVAL; }
  if (P >= ctx->max_ctx) { ctx->err = "prompt_len must be < max_context"; return DEX_E_CAPACITY; }
  const int B = ctx->B, d = ctx->d, H = ctx->H, hd = ctx->hd;
  for (int i = 0; i < B * P; ++i)
    if (prompts[i] < 0 || prompts[i] >= ctx->V) { ctx->err = "prompt token out of range"; return DEX_E_INVAL; }
  const size_t M = (size_t)B * P, es = ctx->es;
  const int G = H / ctx->Hkv;
  // matrix-core prompt attention for bf16 caches; the split kernel otherwise
  const bool mfma_prefill = ctx->dtype == DEX_BF16 && (hd == 64 || hd == 128) && G <= 8;
  const int grp_rows = std::max(1, ATT_MAX_PAIRS / G);
  const int jmax = (P + ATT_SPLIT - 1) / ATT_SPLIT;
  // attention row chunk bounded so its split partials stay below ~512 MiB
  const size_t per_row = (size_t)H * jmax * (hd + 2) * 4;
  size_t chunk = std::max<size_t>(grp_rows, (512ull << 20) / per_row);
  chunk = std::min(chunk, M);
  chunk = (chunk / grp_rows) * grp_rows;
  if (chunk == 0) chunk = grp_rows;

  float *h = nullptr, *part = nullptr, *q = nullptr, *apart = nullptr, *rsc = nullptr;
  void *xb = nullptr, *att = nullptr, *act = nullptr;
  int *tab = nullptr;
  dex_status st = DEX_OK;
  auto A = [&](void **p, size_t bytes) {
    if (st == DEX_OK) st = dalloc(ctx, p, bytes);
  };
  A((void **)&h, M * d * 4);
  A((void **)&part, M * ctx->n_part * 4);
  A(&xb, M * d * es);
  A((void **)&q, M * H * hd * 4);
  A(&att, M * H * hd * es);
  A(&act, M * ctx->F * es);
  A((void **)&rsc, M * 4);
  if (!mfma_prefill) A((void **)&apart, chunk * per_row);
  const size_t n_groups_total = (size_t)B * ((P + grp_rows - 1) / grp_rows);
  const size_t tab_ints = M * 8 + n_groups_total * 4 + 6 * B + 64;
  A((void **)&tab, tab_ints * 4);
  auto cleanup = [&]() {
    dfree(ctx, h); dfree(ctx, part); dfree(ctx, xb); dfree(ctx, q); dfree(ctx, att); dfree(ctx, act);
    dfree(ctx, apart); dfree(ctx, tab); dfree(ctx, rsc);
  };
  if (st != DEX_OK) { cleanup(); return st; }   // nothing changed yet: not poisoned

  // row tables: rows ordered (seq, position)
  std::vector<int> host(tab_ints, 0);
  int *t_seq = host.data(), *t_pos = t_seq + M, *t_entry = t_pos + M, *t_tok = t_entry + M, *t_nc = t_tok + M,
      *t_coff = t_nc + M, *t_bnd = t_coff + M, *t_zero = t_bnd + M;
  int *g_row0 = t_zero + M, *g_nrows = g_row0 + n_groups_total, *g_seq = g_nrows + n_groups_total;
  int *g_rel = g_seq + n_groups_total;
  int *ex_src = g_rel + n_groups_total, *ex_zero = ex_src + B, *ex_cidx = ex_zero + B;
  int *ex_seq = ex_cidx + B, *ex_pos = ex_seq + B;
  for (int s = 0; s < B; ++s)
    for (int p = 0; p < P; ++p) {
      const size_t r = (size_t)s * P + p;
      t_seq[r] = s; t_pos[r] = p; t_entry[r] = p; t_tok[r] = prompts[r]; t_nc[r] = p + 1;
      t_coff[r] = 0; t_bnd[r] = 0; t_zero[r] = 0;
    }
  std::vector<int> gr0, gnr, gsq;
  for (int s = 0; s < B; ++s)
    for (int p = 0; p < P; p += grp_rows) {
      gr0.push_back(s * P + p);
      gnr.push_back(std::min(grp_rows, P - p));
      gsq.push_back(s);
    }
  const int ng = (int)gr0.size();
  std::copy(gr0.begin(), gr0.end(), g_row0);
  std::copy(gnr.begin(), gnr.end(), g_nrows);
  std::copy(gsq.begin(), gsq.end(), g_seq);
  // attention chunks: runs of whole groups holding at most `chunk` rows
  std::vector<std::array<int, 4>> chunks;   // first group, groups, first row, rows
  for (int g = 0; g < ng;) {
    const int c0 = gr0[g];
    int e = g, rows_in = 0;
    while (e < ng && (rows_in + gnr[e] <= (int)chunk || e == g)) { rows_in += gnr[e]; ++e; }
    for (int i = g; i < e; ++i) g_rel[i] = gr0[i] - c0;
    chunks.push_back({g, e - g, c0, rows_in});
    g = e;
  }
  for (int s = 0; s < B; ++s) {
    ex_src[s] = s * P + P - 1; ex_zero[s] = 0; ex_cidx[s] = 0; ex_seq[s] = s; ex_pos[s] = P - 1;
  }
  HIPCHK(hipMemcpyAsync(tab, host.data(), tab_ints * 4, hipMemcpyHostToDevice, ctx->stream));
  const int *d_seq = tab, *d_pos = tab + M, *d_entry = d_pos + M, *d_tok = d_entry + M, *d_nc = d_tok + M,
            *d_coff = d_nc + M, *d_zero = d_coff + 2 * M;
  const int *d_g0 = d_zero + M, *d_gn = d_g0 + n_groups_total, *d_gs = d_gn + n_groups_total;
  const int *d_grel = d_gs + n_groups_total;
  const int *d_exsrc = d_grel + n_groups_total, *d_exzero = d_exsrc + B;
  const int *d_exseq = d_exzero + 2 * B, *d_expos = d_exseq + B;

  {
    PrepArgs p{};
    p.M = (int)M; p.d = d; p.n_part = ctx->n_part; p.embed_rows = (int)M; p.row_tok = d_tok; p.embed = ctx->embed;
    p.g = (const float *)LW(ctx, 0, DEX_P_ATTN_NORM); p.h = h; p.part = part; p.xb = xb;
    HIPCHK(launch_prep(ctx->dtype, p, ctx->stream));
  }
  const size_t layer_kv = (size_t)B * ctx->Hkv * ctx->E * hd * es;
  // many prompt rows: the M-tiled kernel (bf16; a normed GEMM first gets
  // its row scales); the decode kernel otherwise
  auto prefill_gemm = [&](int epi, const GemmArgs &a) -> hipError_t {
    if (ctx->dtype == DEX_BF16 && a.M > 64) {
      GemmArgs t = a;
      t.row_rsc = a.part != nullptr ? rsc : nullptr;
      if (gemm_tiled_supported(epi, t)) {
        if (t.row_rsc != nullptr) {
          const hipError_t e = launch_row_scale(a.part, a.n_part, a.M, a.inv_d, a.eps, rsc, ctx->stream);
          if (e != hipSuccess) return e;
        }
        return launch_gemm_tiled(epi, t, ctx->stream);
      }
    }
    return launch_gemm(ctx->dtype, epi, a, 1, ctx->stream);
  };
  for (int l = 0; l < ctx->L; ++l) {
    const float alpha = ctx->rscale * (float)(l + 1) / (float)ctx->L;
    {
      GemmArgs a{};
      a.wp = ctx->p_qkv[l]; a.nsteps_w = ctx->ns_d;
      a.N = (H + 2 * ctx->Hkv) * hd; a.K = d; a.x = xb; a.ldx = d; a.M = (int)M;
      a.part = part; a.n_part = ctx->n_part; a.inv_d = 1.0f / d; a.eps = ctx->eps;
      a.out = q; a.ld_out = H * hd;
      a.kc = (char *)ctx->kc + l * layer_kv; a.vc = (char *)ctx->vc + l * layer_kv;
      a.kv_entries = ctx->E; a.n_heads = H; a.n_kv_heads = ctx->Hkv; a.head_dim = hd;
      a.row_seq = d_seq; a.row_pos = d_pos; a.row_entry = d_entry; a.rope = ctx->rope;
      HIPCHK(prefill_gemm(EPI_QKV, a));
    }
    if (mfma_prefill) {
      PrefillAttnArgs a{};
      a.q = q; a.ldq = H * hd;
      a.kc = (char *)ctx->kc + l * layer_kv; a.vc = (char *)ctx->vc + l * layer_kv;
      a.kv_entries = ctx->E; a.n_kv_heads = ctx->Hkv; a.n_heads = H; a.head_dim = hd; a.batch = B;
      a.prompt_len = P; a.scale = 1.0f / std::sqrt((float)hd); a.out = att; a.ld_out = H * hd;
      HIPCHK(launch_prefill_attention(a, ctx->stream));
    } else for (const auto &ch : chunks) {
      const int g_first = ch[0], g_cnt = ch[1], c0 = ch[2], cn = ch[3];
      AttnArgs a{};
      a.q = q + (size_t)c0 * H * hd; a.ldq = H * hd;
      a.kc = (char *)ctx->kc + l * layer_kv; a.vc = (char *)ctx->vc + l * layer_kv;
      a.kv_entries = ctx->E; a.n_kv_heads = ctx->Hkv; a.n_heads = H; a.head_dim = hd; a.batch = B;
      a.grp_row0 = d_grel + g_first; a.grp_nrows = d_gn + g_first; a.grp_seq = d_gs + g_first;
      a.row_pos = d_pos + c0; a.row_nc = d_nc + c0; a.row_chain_off = d_coff + c0; a.chain = d_zero;
      a.row_seq = d_seq + c0; a.n_rows = cn;
      a.part = apart; a.stat = split_stats(apart, cn, H, jmax, hd);
      a.jmax = jmax; a.n_splits = jmax; a.scale = 1.0f / std::sqrt((float)hd);
      HIPCHK(launch_attention(ctx->dtype, a, g_cnt, ctx->stream));
      CombineArgs cb{};
      cb.part = apart; cb.stat = split_stats(apart, cn, H, jmax, hd);
      cb.row_pos = d_pos + c0; cb.jmax = jmax; cb.n_heads = H; cb.head_dim = hd;
      cb.out = (char *)att + (size_t)c0 * H * hd * es; cb.ld_out = H * hd;
      HIPCHK(launch_combine(ctx->dtype, cb, cn, ctx->stream));
    }
    {
      GemmArgs a{};
      a.wp = ctx->p_o[l]; a.nsteps_w = ctx->ns_hhd; a.N = d; a.K = H * hd; a.x = att; a.ldx = H * hd; a.M = (int)M;
      a.h = h; a.ld_h = d; a.alpha = alpha; a.g_next = (const float *)LW(ctx, l, DEX_P_FFN_NORM); a.xb = xb;
      a.part_out = part; a.n_part_out = ctx->n_part;
      HIPCHK(prefill_gemm(EPI_RESID, a));
    }
    {
      GemmArgs a{};
      a.wp = ctx->p_gu[l]; a.nsteps_w = ctx->ns_d; a.N = ctx->F; a.K = d;
      a.x = xb; a.ldx = d; a.M = (int)M; a.part = part; a.n_part = ctx->n_part; a.inv_d = 1.0f / d;
      a.eps = ctx->eps; a.act = act; a.ld_act = ctx->F;
      HIPCHK(prefill_gemm(EPI_SWIGLU, a));
    }
    {
      const bool last = l == ctx->L - 1;
      GemmArgs a{};
      a.wp = ctx->p_down[l]; a.nsteps_w = ctx->ns_F; a.N = d; a.K = ctx->F; a.x = act; a.ldx = ctx->F; a.M = (int)M;
      a.h = h; a.ld_h = d; a.alpha = alpha;
      a.g_next = last ? nullptr : (const float *)LW(ctx, l + 1, DEX_P_ATTN_NORM);
      a.xb = last ? nullptr : xb; a.part_out = part; a.n_part_out = ctx->n_part;
      HIPCHK(prefill_gemm(EPI_RESID, a));
    }
  }
  // y_0: final-depth exit head at the last prompt position of every sequence
  dex_status es2 = run_exit(ctx, B, d_exsrc, h, part, d_exzero, d_exzero, nullptr, nullptr, d_exseq, d_expos, nullptr,
                            nullptr);
  if (es2 != DEX_OK) { cleanup(); return fail(ctx, es2); }
  HIPCHK(hipMemcpyAsync(ctx->res_host, ctx->u_dev, B * 4, hipMemcpyDeviceToHost, ctx->stream));
  HIPCHK(hipStreamSynchronize(ctx->stream));
  cleanup();
  harvest_timing(ctx);
  for (int s = 0; s < B; ++s) {
    Seq &q2 = ctx->seqs[s];
    q2.committed.assign(prompts + (size_t)s * P, prompts + (size_t)(s + 1) * P);
    const int y0 = ctx->res_host[s];
    q2.committed.push_back(y0);
    first[s] = y0;
    q2.slots.clear();
    Slot a;
    a.x = y0; a.pos = P; a.u.clear(); a.child.assign(ctx->N, -1);
    q2.slots.push_back(a);
    q2.half = 0;
    q2.active = (int)q2.committed.size() < ctx->max_ctx;
    q2.last_map.clear(); q2.last_fresh = -1; q2.last_committed_pos = -1;
  }
  ctx->prefilled = true;
  ctx->rounds = 0;
  return DEX_OK;
}

dex_status dex_step(dex_ctx *ctx, int32_t *committed_out, dex_step_info *info) {
  if (!ctx) return DEX_E_INVAL;
  if (ctx->poisoned) { ctx->err = "context poisoned by an earlier failure"; return DEX_E_STATE; }
  if (!ctx->prefilled) { ctx->err = "dex_step before dex_prefill"; return DEX_E_STATE; }
  if (!committed_out) { ctx->err = "committed is NULL"; return DEX_E_INVAL; }
  const int N = ctx->N, B = ctx->B;
  const auto t_call = std::chrono::steady_clock::now();
  for (int s = 0; s < B; ++s) committed_out[s] = -1;
  bool any = false;
  for (auto &s : ctx->seqs) any |= s.active;
  if (!any) { ctx->err = "every sequence reached max_context"; return DEX_E_CAPACITY; }

  // ---------------------------------------------------------------- plan
  std::vector<Row> rows;            // priority order within each sequence
  std::vector<int> q_start(B, -1);
  for (int si = 0; si < B; ++si) {
    Seq &s = ctx->seqs[si];
    if (!s.active) continue;
    q_start[si] = s.slots[0].c;
    std::vector<Item> items = plan_items(PlanRule{ctx->N, ctx->W, ctx->decs, ctx->max_ctx}, s);
    for (const Item &it : items) {
      if (it.kind == 0) {
        rows.push_back({si, it.slot, s.slots[it.slot].c});
      } else {
        if ((int)s.slots.size() >= ctx->S) return fail_mid_round(ctx, "lattice slot capacity exceeded", DEX_E_CAPACITY);
        Slot ns;
        ns.x = s.slots[it.slot].u[it.f];
        ns.pos = s.slots[it.slot].pos + 1;
        ns.parent = it.slot;
        ns.fork_stage = it.f;
        ns.child.assign(N, -1);
        s.slots.push_back(ns);
        const int ni = (int)s.slots.size() - 1;
        s.slots[it.slot].child[it.f] = ni;
        rows.push_back({si, ni, 0});
      }
    }
  }
  // stage-major order, then sequence, then priority (stable)
  std::stable_sort(rows.begin(), rows.end(), [](const Row &a, const Row &b) {
    if (a.stage != b.stage) return a.stage < b.stage;
    return a.seq < b.seq;
  });
  const int R = (int)rows.size();
  if (R > ctx->R_max) return fail_mid_round(ctx, "round rows exceed capacity", DEX_E_CAPACITY);

  // ------------------------------------------------------- row tables
  int *T = ctx->tab_host;
  int *t_seq = T, *t_pos = T + R, *t_entry = T + 2 * R, *t_bnd = T + 3 * R, *t_tok = T + 4 * R,
      *t_nc = T + 5 * R, *t_coff = T + 6 * R, *t_maskn = T + 7 * R, *t_cidx = T + 8 * R;
  int *t_mask = T + 9 * R;                 // [R][N]
  int *t_chain = t_mask + R * N;           // [R * CH_MAX]
  int *t_g0 = t_chain + R * ctx->CH_MAX;   // groups (stage-local row0), up to R
  int *t_gn = t_g0 + R, *t_gs = t_gn + R;
  int *t_gnc = t_gs + R;                   // committed prefix length of each group's rows
  int *t_rcommit = t_gnc + R;              // [R] commit slot of a row completing its anchor, else -1
  std::vector<int> stage_r0(N + 1, 0), stage_g0(N + 1, 0);
  int chain_used = 0, ngroups = 0;
  const int G = ctx->H / ctx->Hkv;
  const int grp_rows = std::max(1, ATT_MAX_PAIRS / G);
  for (int r = 0; r < R; ++r) {
    const Row &rw = rows[r];
    const Seq &s = ctx->seqs[rw.seq];
    const Slot &sl = s.slots[rw.slot];
    t_seq[r] = rw.seq;
    t_pos[r] = sl.pos;
    t_entry[r] = slot_entry(ctx, s, rw.slot);
    t_bnd[r] = slot_global(ctx, rw.seq, s, rw.slot);
    t_tok[r] = sl.x;
    t_nc[r] = (int)s.committed.size() - 1;
    t_coff[r] = chain_used;
    std::vector<int> anc = ancestors(s, rw.slot);
    if ((int)anc.size() + 1 > ctx->CH_MAX) return fail_mid_round(ctx, "lattice chain too deep", DEX_E_CAPACITY);
    for (int a : anc) t_chain[chain_used++] = slot_entry(ctx, s, a);
    t_chain[chain_used++] = slot_entry(ctx, s, rw.slot);
    // DECS mask: tokens proposed by shallower nodes of this slot chain,
    // except the anchor's final-depth node
    int nm = 0;
    if (ctx->decs && !(rw.slot == 0 && rw.stage == N - 1))
      for (int j = 0; j < rw.stage; ++j) t_mask[r * N + nm++] = sl.u[j];
    t_maskn[r] = nm;
    t_cidx[r] = t_bnd[r] * N + rw.stage;
    stage_r0[rw.stage + 1] = r + 1;
  }
  for (int k = 1; k <= N; ++k) stage_r0[k] = std::max(stage_r0[k], stage_r0[k - 1]);
  // attention row groups per stage: consecutive rows of one sequence
  for (int k = 0; k < N; ++k) {
    stage_g0[k] = ngroups;
    for (int r = stage_r0[k]; r < stage_r0[k + 1];) {
      int e = r;
      // (the rows of a group share their committed prefix: the attention
      // kernels rely on it)
      while (e < stage_r0[k + 1] && rows[e].seq == rows[r].seq && t_nc[e] == t_nc[r] && e - r < grp_rows) ++e;
      t_g0[ngroups] = r - stage_r0[k];
      t_gn[ngroups] = e - r;
      t_gs[ngroups] = rows[r].seq;
      t_gnc[ngroups] = t_nc[r];
      ++ngroups;
      r = e;
    }
  }
  stage_g0[N] = ngroups;
  std::vector<int> commit_seqs;
  for (int r = 0; r < R; ++r) t_rcommit[r] = -1;
  for (int si = 0; si < B; ++si) {
    Seq &s = ctx->seqs[si];
    if (s.active && s.slots[0].c == N - 1) {
      for (int r = 0; r < R; ++r)
        if (rows[r].seq == si && rows[r].slot == 0) t_rcommit[r] = (int)commit_seqs.size();
      commit_seqs.push_back(si);
    }
  }
  const size_t tab_ints = (size_t)(t_rcommit - T) + R;
  if (tab_ints > ctx->tab_cap) return fail_mid_round(ctx, "row table overflow", DEX_E_CAPACITY);
  hipEvent_t *rt = ctx->round_timing ? ctx->rt_ev[ctx->rt_cur] : nullptr;
  if (rt) {
    ctx->rt_ms[6] += std::chrono::duration<double, std::milli>(std::chrono::steady_clock::now() - t_call).count();
    HIPCHK(hipEventRecord(rt[0], ctx->stream));
  }
  HIPCHK(hipMemcpyAsync(ctx->tab_dev, T, tab_ints * 4, hipMemcpyHostToDevice, ctx->stream));
  if (rt) HIPCHK(hipEventRecord(rt[1], ctx->stream));
  const int *D = ctx->tab_dev;
  auto dptr = [&](const int *hp) { return D + (hp - T); };

  // ------------------------------------------------------------ sweep
  // The stages of a round are independent: each row reads the boundary
  // state its slot reached in an earlier round, writes its own slot's, and
  // touches the key/value cache only in its own stage's layers.  Each stage
  // works in its own row range of the scratch buffers, so the stages can be
  // spread over the lanes; the exit heads wait for all of them.  (Per-kernel
  // timing keeps everything on one stream.)
  const bool multi = ctx->n_lanes > 1 && !ctx->timing;

  if (multi) {
    HIPCHK(hipEventRecord(ctx->fork_ev, ctx->stream));
    for (int i = 1; i < ctx->n_lanes; ++i) HIPCHK(hipStreamWaitEvent(ctx->lane_st[i], ctx->fork_ev, 0));
  }
  // stages with rows go round-robin over the lanes
  // (grouped: contiguous runs of them, one per lane, so that each lane's rows
  // are consecutive)
  std::vector<int> stage_lane(N, -1);
  if (ctx->grouped) {
    std::vector<int> act;
    for (int k = 0; k < N; ++k)
      if (stage_r0[k + 1] > stage_r0[k]) act.push_back(k);
    const int na = (int)act.size(), nl = multi ? std::min(ctx->n_lanes, na) : 1;
    for (int i = 0; i < na; ++i) stage_lane[act[i]] = i * nl / na;
  } else {
    int lane_next = 0;
    for (int k = 0; k < N; ++k)
      if (stage_r0[k + 1] > stage_r0[k]) stage_lane[k] = multi ? lane_next++ % ctx->n_lanes : 0;
  }
  struct LaneSum {
    int layers = 0, row_layers = 0;
    double attn_bytes = 0.0;
  };
  std::vector<LaneSum> lane_sum(ctx->n_lanes);
  // a stage's tables, its share of the round's sums, and the launch that
  // gives its rows their first RMSNorm input (from the embedding or the
  // boundary state their slot reached)
  auto stage_prologue = [&](int k, StageTables &t, hipStream_t lst, bool prep) -> dex_status {
    const int r0 = stage_r0[k], M = stage_r0[k + 1] - r0;
    LaneSum &acc = lane_sum[stage_lane[k]];
    const std::vector<int> &ls = ctx->stage_layers[k];
    acc.layers += (int)ls.size();
    acc.row_layers += M * (int)ls.size();
    t = StageTables{};
    t.seq = dptr(t_seq) + r0; t.pos = dptr(t_pos) + r0; t.entry = dptr(t_entry) + r0; t.bnd = dptr(t_bnd) + r0;
    t.tok = dptr(t_tok) + r0; t.nc = dptr(t_nc) + r0; t.chain_off = dptr(t_coff) + r0; t.chain = dptr(t_chain);
    t.g_row0 = dptr(t_g0) + stage_g0[k]; t.g_nrows = dptr(t_gn) + stage_g0[k]; t.g_seq = dptr(t_gs) + stage_g0[k];
    t.g_nc = dptr(t_gnc) + stage_g0[k];
    t.n_groups = stage_g0[k + 1] - stage_g0[k];
    t.attn_bytes = 0.0;
    int stage_maxpos = 0;
    for (int g = stage_g0[k]; g < stage_g0[k + 1]; ++g) {
      int mp = 0;
      for (int r = stage_r0[k] + t_g0[g]; r < stage_r0[k] + t_g0[g] + t_gn[g]; ++r) mp = std::max(mp, t_pos[r]);
      t.attn_bytes += (double)(mp + 1) * 2.0 * ctx->Hkv * ctx->hd * ctx->es;
      stage_maxpos = std::max(stage_maxpos, mp);
    }
    t.n_splits = std::min(ctx->jmax, stage_maxpos / ATT_SPLIT + 1);
    t.attn_bytes += (double)M * ctx->H * ctx->hd * (4.0 + ctx->es);
    acc.attn_bytes += t.attn_bytes * (double)ls.size();
    if (prep) {
      PrepArgs p{};
      p.M = M; p.d = ctx->d; p.n_part = ctx->n_part; p.embed_rows = (k == 0) ? M : 0;
      p.row_tok = t.tok; p.row_src = t.bnd; p.embed = ctx->embed; p.bnd_h = ctx->bnd_h; p.bnd_part = ctx->bnd_part;
      p.g = (const float *)LW(ctx, ls.front(), DEX_P_ATTN_NORM);
      p.h = ctx->h_w + (size_t)r0 * ctx->d; p.part = ctx->part_w + (size_t)r0 * ctx->n_part;
      p.xb = (char *)ctx->xb_w + (size_t)r0 * ctx->d * ctx->es;
      TimedLaunch tl(ctx, 7, 0.0);
      HIPCHK(launch_prep(ctx->dtype, p, lst));
    }
    return DEX_OK;
  };
  auto run_stage = [&](int k) -> dex_status {
    const int r0 = stage_r0[k], M = stage_r0[k + 1] - r0;
    const hipStream_t lst = multi ? ctx->lane_st[stage_lane[k]] : ctx->stream;
    const std::vector<int> &ls = ctx->stage_layers[k];
    StageTables t{};
    const dex_status ps = stage_prologue(k, t, lst, true);
    if (ps != DEX_OK) return ps;
    return run_layers(ctx, lst, ls.front(), ls.back(), M, t, ctx->h_w + (size_t)r0 * ctx->d,
                      ctx->part_w + (size_t)r0 * ctx->n_part,
                      (char *)ctx->xb_w + (size_t)r0 * ctx->d * ctx->es,
                      ctx->q_w + (size_t)r0 * ctx->H * ctx->hd,
                      (char *)ctx->att_w + (size_t)r0 * ctx->H * ctx->hd * ctx->es,
                      (char *)ctx->act_w + (size_t)r0 * ctx->F * ctx->es,
                      ctx->attn_part + (size_t)r0 * ctx->H * ctx->jmax * (ctx->hd + 2), ctx->jmax,
                      true, t.bnd);
  };
  // grouped: a lane's stages in step, layer step j of every one of them that
  // has one in a single launch per kernel (segments in stage order, whose
  // rows are consecutive in the round's buffers)
  auto run_grouped = [&](int lane) -> dex_status {
    const int d = ctx->d, H = ctx->H, Hkv = ctx->Hkv, hd = ctx->hd, F = ctx->F, jmax = ctx->jmax;
    const size_t layer_kv = (size_t)B * Hkv * ctx->E * hd * ctx->es;
    const hipStream_t st = multi ? ctx->lane_st[lane] : ctx->stream;
    std::vector<int> ks;
    std::vector<StageTables> tabs(N);
    size_t depth = 0;
    for (int k = 0; k < N; ++k) {
      if (stage_lane[k] != lane) continue;
      const dex_status ps = stage_prologue(k, tabs[k], st, false);
      if (ps != DEX_OK) return ps;
      ks.push_back(k);
      depth = std::max(depth, ctx->stage_layers[k].size());
    }
    // the stages' first RMSNorm inputs: one launch per run of at most
    // MAX_SEGS stages (a lane's stages are consecutive among those with
    // rows, so their rows are consecutive; stage 0, if present, comes first)
    for (size_t i0 = 0; i0 < ks.size(); i0 += MAX_SEGS) {
      const size_t c = std::min<size_t>(MAX_SEGS, ks.size() - i0);
      const int ra = stage_r0[ks[i0]], rb = stage_r0[ks[i0 + c - 1] + 1];
      PrepArgs p{};
      p.M = rb - ra; p.d = ctx->d; p.n_part = ctx->n_part;
      p.embed_rows = ks[i0] == 0 ? stage_r0[1] - stage_r0[0] : 0;
      p.row_tok = dptr(t_tok) + ra; p.row_src = dptr(t_bnd) + ra;
      p.embed = ctx->embed; p.bnd_h = ctx->bnd_h; p.bnd_part = ctx->bnd_part;
      p.n_seg = (int)c;
      for (size_t i = 0; i < c; ++i) {
        const int k = ks[i0 + i];
        p.seg_end[i] = stage_r0[k + 1] - ra;
        p.seg_g[i] = (const float *)LW(ctx, ctx->stage_layers[k].front(), DEX_P_ATTN_NORM);
      }
      p.g = p.seg_g[0];
      p.h = ctx->h_w + (size_t)ra * ctx->d; p.part = ctx->part_w + (size_t)ra * ctx->n_part;
      p.xb = (char *)ctx->xb_w + (size_t)ra * ctx->d * ctx->es;
      TimedLaunch tl(ctx, 7, 0.0);
      HIPCHK(launch_prep(ctx->dtype, p, st));
    }
    // split records of every row of the round: [R][H][jmax][hd], then the
    // statistics
    float *stat_all = split_stats(ctx->attn_part, R, H, jmax, hd);
    const size_t rec_row = (size_t)H * jmax * hd * ctx->es;     // record bytes per row
    std::vector<int> on, lay;
    std::vector<GemmSeg> gs(ks.size());
    std::vector<AttnSeg> as(ks.size());
    for (size_t j = 0; j < depth; ++j) {
      on.clear();
      lay.clear();
      for (int k : ks)
        if (j < ctx->stage_layers[k].size()) {
          on.push_back(k);
          lay.push_back(ctx->stage_layers[k][j]);
        }
      const int n = (int)on.size();
      auto seg_rows = [&](GemmSeg &g, int i) {
        g.r0 = stage_r0[on[i]];
        g.M = stage_r0[on[i] + 1] - g.r0;
      };
      // QKV
      {
        GemmArgs a{};
        a.nsteps_w = ctx->ns_d; a.N = (H + 2 * Hkv) * hd; a.K = d;
        a.x = ctx->xb_w; a.ldx = d;
        a.part = ctx->part_w; a.n_part = ctx->n_part; a.inv_d = 1.0f / d; a.eps = ctx->eps;
        a.out = ctx->q_w; a.ld_out = H * hd;
        a.kv_entries = ctx->E; a.n_heads = H; a.n_kv_heads = Hkv; a.head_dim = hd;
        a.row_seq = dptr(t_seq); a.row_pos = dptr(t_pos); a.row_entry = dptr(t_entry); a.rope = ctx->rope;
        double bytes = 0.0;
        for (int i = 0; i < n; ++i) {
          const int l = lay[i];
          GemmSeg &g = gs[i];
          g = GemmSeg{};
          g.wp = ctx->p_qkv[l];
          g.kc = (char *)ctx->kc + l * layer_kv;
          g.vc = (char *)ctx->vc + l * layer_kv;
          seg_rows(g, i);
          bytes += wbytes(ctx, (double)a.N * d + (double)g.M * d + 2.0 * g.M * Hkv * hd) + 4.0 * g.M * H * hd;
        }
        TimedLaunch tl(ctx, 0, bytes);
        HIPCHK(launch_gemm_seg(ctx->dtype, EPI_QKV, a, gs.data(), n, st));
      }
      // attention
      {
        AttnArgs a{};
        a.q = ctx->q_w; a.ldq = H * hd;
        a.kv_entries = ctx->E; a.n_kv_heads = Hkv; a.n_heads = H; a.head_dim = hd; a.batch = B;
        a.grp_row0 = dptr(t_g0); a.grp_nrows = dptr(t_gn); a.grp_seq = dptr(t_gs); a.grp_nc = dptr(t_gnc);
        a.row_pos = dptr(t_pos); a.row_nc = dptr(t_nc); a.row_chain_off = dptr(t_coff); a.chain = dptr(t_chain);
        a.row_seq = dptr(t_seq);
        a.part = ctx->attn_part; a.stat = stat_all;
        a.jmax = jmax; a.scale = 1.0f / std::sqrt((float)hd);
        double bytes = 0.0;
        for (int i = 0; i < n; ++i) {
          const int k = on[i], l = lay[i];
          AttnSeg &g = as[i];
          g.kc = (char *)ctx->kc + l * layer_kv;
          g.vc = (char *)ctx->vc + l * layer_kv;
          g.r0 = stage_r0[k];
          g.M = stage_r0[k + 1] - stage_r0[k];
          g.g0 = stage_g0[k];
          g.n_groups = tabs[k].n_groups;
          g.n_splits = tabs[k].n_splits;
          bytes += tabs[k].attn_bytes;
        }
        TimedLaunch tl(ctx, 1, bytes);
        HIPCHK(launch_attention_seg(ctx->dtype, a, as.data(), n, st));
      }
      // split combine over each run of consecutive rows
      for (int i = 0; i < n;) {
        const int ra = stage_r0[on[i]];
        int rb = stage_r0[on[i] + 1], e = i + 1;
        while (e < n && stage_r0[on[e]] == rb) rb = stage_r0[on[e++] + 1];
        CombineArgs c{};
        c.part = (char *)ctx->attn_part + ra * rec_row;
        c.stat = stat_all + (size_t)ra * H * jmax * 2;
        c.row_pos = dptr(t_pos) + ra; c.jmax = jmax; c.n_heads = H; c.head_dim = hd;
        c.out = (char *)ctx->att_w + (size_t)ra * H * hd * ctx->es; c.ld_out = H * hd;
        TimedLaunch tl(ctx, 2, 0.0);
        HIPCHK(launch_combine(ctx->dtype, c, rb - ra, st));
        i = e;
      }
      // O projection + residual
      {
        GemmArgs a{};
        a.nsteps_w = ctx->ns_hhd; a.N = d; a.K = H * hd;
        a.x = ctx->att_w; a.ldx = H * hd;
        a.h = ctx->h_w; a.ld_h = d; a.xb = ctx->xb_w;
        a.part_out = ctx->part_w; a.n_part_out = ctx->n_part;
        double bytes = 0.0;
        for (int i = 0; i < n; ++i) {
          const int l = lay[i];
          GemmSeg &g = gs[i];
          g = GemmSeg{};
          g.wp = ctx->p_o[l];
          g.alpha = ctx->rscale * (float)(l + 1) / (float)ctx->L;
          g.g_next = (const float *)LW(ctx, l, DEX_P_FFN_NORM);
          seg_rows(g, i);
          bytes += wbytes(ctx, (double)d * H * hd + (double)g.M * H * hd + (double)g.M * d) + 8.0 * g.M * d;
        }
        TimedLaunch tl(ctx, 3, bytes);
        HIPCHK(launch_gemm_seg(ctx->dtype, EPI_RESID, a, gs.data(), n, st));
      }
      // gate/up + SiLU
      {
        GemmArgs a{};
        a.nsteps_w = ctx->ns_d; a.N = F; a.K = d;
        a.x = ctx->xb_w; a.ldx = d;
        a.part = ctx->part_w; a.n_part = ctx->n_part; a.inv_d = 1.0f / d; a.eps = ctx->eps;
        a.act = ctx->act_w; a.ld_act = F;
        double bytes = 0.0;
        for (int i = 0; i < n; ++i) {
          GemmSeg &g = gs[i];
          g = GemmSeg{};
          g.wp = ctx->p_gu[lay[i]];
          seg_rows(g, i);
          bytes += wbytes(ctx, 2.0 * F * d + (double)g.M * d + (double)g.M * F);
        }
        TimedLaunch tl(ctx, 4, bytes);
        HIPCHK(launch_gemm_seg(ctx->dtype, EPI_SWIGLU, a, gs.data(), n, st));
      }
      // down + residual; a stage's last layer writes its rows' boundary state
      {
        GemmArgs a{};
        a.nsteps_w = ctx->ns_F; a.N = d; a.K = F;
        a.x = ctx->act_w; a.ldx = F;
        a.h = ctx->h_w; a.ld_h = d; a.xb = ctx->xb_w;
        a.part_out = ctx->part_w; a.n_part_out = ctx->n_part;
        a.bnd_h = ctx->bnd_h; a.bnd_part = ctx->bnd_part;
        double bytes = 0.0;
        for (int i = 0; i < n; ++i) {
          const int k = on[i], l = lay[i];
          const bool last = (j + 1 == ctx->stage_layers[k].size());
          GemmSeg &g = gs[i];
          g = GemmSeg{};
          g.wp = ctx->p_down[l];
          g.alpha = ctx->rscale * (float)(l + 1) / (float)ctx->L;
          g.g_next = last ? nullptr : (const float *)LW(ctx, l + 1, DEX_P_ATTN_NORM);
          g.row_bnd = last ? tabs[k].bnd : nullptr;
          seg_rows(g, i);
          bytes += wbytes(ctx, (double)d * F + (double)g.M * F + (double)g.M * d) + 8.0 * g.M * d;
        }
        TimedLaunch tl(ctx, 5, bytes);
        HIPCHK(launch_gemm_seg(ctx->dtype, EPI_RESID, a, gs.data(), n, st));
      }
    }
    return DEX_OK;
  };
  // a lane's stages, in stage order
  auto run_lane = [&](int lane) -> dex_status {
    if (ctx->grouped) return run_grouped(lane);
    for (int k = 0; k < N; ++k)
      if (stage_lane[k] == lane) {
        const dex_status st = run_stage(k);
        if (st != DEX_OK) return st;
      }
    return DEX_OK;
  };
  if (multi && !ctx->lane_threads.empty()) {
    // each lane from its own thread (lane 0: this one)
    ctx->lane_fn = run_lane;
    const int64_t ticket = ctx->lane_ticket.load(std::memory_order_relaxed) + 1;
    {
      std::lock_guard<std::mutex> lk(ctx->lane_mu);
      ctx->lane_ticket.store(ticket, std::memory_order_release);
    }
    ctx->lane_cv.notify_all();
    dex_status rs = run_lane(0);
    for (int i = 1; i < ctx->n_lanes; ++i) {
      while (ctx->lane_done[i].load(std::memory_order_acquire) != ticket) std::this_thread::yield();
      if (rs == DEX_OK && ctx->lane_status[i] != DEX_OK) {
        rs = ctx->lane_status[i];
        ctx->err = ctx->lane_err[i];
      }
    }
    ctx->lane_fn = nullptr;
    if (rs != DEX_OK) return fail(ctx, rs);
  } else {
    for (int lane = 0; lane < ctx->n_lanes; ++lane) {
      const dex_status rs = run_lane(lane);
      if (rs != DEX_OK) return fail(ctx, rs);
    }
  }
  int layers_streamed = 0, row_layers = 0;
  double attn_bytes = 0.0;
  for (const LaneSum &ls : lane_sum) {
    layers_streamed += ls.layers;
    row_layers += ls.row_layers;
    attn_bytes += ls.attn_bytes;
  }
  if (multi) {
    for (int i = 1; i < ctx->n_lanes; ++i) {
      HIPCHK(hipEventRecord(ctx->lane_ev[i], ctx->lane_st[i]));
      HIPCHK(hipStreamWaitEvent(ctx->stream, ctx->lane_ev[i], 0));
    }
  }
  // ---------------------------------------------------- exit + commit
  if (rt) HIPCHK(hipEventRecord(rt[2], ctx->stream));
  dex_status xs = run_exit(ctx, R, dptr(t_bnd), ctx->bnd_h, ctx->bnd_part, dptr(t_maskn), dptr(t_mask),
                           dptr(t_cidx), ctx->cand, dptr(t_seq), dptr(t_pos), stage_r0.data(), dptr(t_rcommit));
  if (xs != DEX_OK) return fail(ctx, xs);
  if (rt) HIPCHK(hipEventRecord(rt[3], ctx->stream));
  // candidates, then (token, k*) of the committing sequences, in one copy
  HIPCHK(hipMemcpyAsync(ctx->res_host, ctx->u_dev, (R + 2 * commit_seqs.size()) * 4, hipMemcpyDeviceToHost,
                        ctx->stream));
  if (rt) HIPCHK(hipEventRecord(rt[4], ctx->stream));
  HIPCHK(hipStreamSynchronize(ctx->stream));
  if (rt) {
    // this round's device phases; the previous round's collapse (its host
    // commit handling and the gather) and the gap before this round
    float ms = 0.f;
    for (int i = 0; i < 4; ++i) {
      HIPCHK(hipEventElapsedTime(&ms, rt[i], rt[i + 1]));
      ctx->rt_ms[i] += ms;
    }
    if (ctx->rt_prev) {
      hipEvent_t *pv = ctx->rt_ev[1 - ctx->rt_cur];
      HIPCHK(hipEventElapsedTime(&ms, pv[4], pv[5]));
      ctx->rt_ms[4] += ms;
      HIPCHK(hipEventElapsedTime(&ms, pv[5], rt[0]));
      ctx->rt_ms[5] += ms;
    }
    ctx->rt_rounds += 1;
  }
  harvest_timing(ctx);
  ctx->rounds += 1;

  // --------------------------------------------------- insert candidates
  for (int r = 0; r < R; ++r) {
    Slot &sl = ctx->seqs[rows[r].seq].slots[rows[r].slot];
    sl.u.push_back(ctx->res_host[r]);
    sl.c += 1;
  }
  if (info) {
    std::memset(info, 0, sizeof(*info));
    info->n_rows = R;
    for (int r = 0; r < R && r < DEX_MAX_ROWS; ++r) {
      info->rows_per_stage[rows[r].stage] += 1;
      info->row_seq[r] = rows[r].seq;
      info->row_slot[r] = rows[r].slot;
      info->row_stage[r] = rows[r].stage;
      info->row_pos[r] = ctx->seqs[rows[r].seq].slots[rows[r].slot].pos;
      info->row_token[r] = ctx->res_host[r];
    }
    info->layers_streamed = layers_streamed;
    info->row_layers = row_layers;
    for (int s = 0; s < B; ++s) { info->q[s] = q_start[s]; info->kstar[s] = -1; }
    info->rounds_total = ctx->rounds;
    info->attn_bytes = attn_bytes;
  }
  // ------------------------------------------------- commit + collapse
  int njobs = 0;
  int *J = ctx->job_host;
  for (size_t ci = 0; ci < commit_seqs.size(); ++ci) {
    const int si = commit_seqs[ci];
    Seq &s = ctx->seqs[si];
    const Slot A = s.slots[0];
    const int y = ctx->res_host[R + 2 * ci], kstar = ctx->res_host[R + 2 * ci + 1];
    // the host's own reading of the same rule must agree with the device
    int kh = N - 1;
    for (int j = 0; j < N - 1; ++j)
      if (A.u[j] == A.u[N - 1]) { kh = j; break; }
    if (A.c != N || y != A.u[N - 1] || kstar != kh)
      return fail_mid_round(ctx, "commit mismatch between device and host lattice", DEX_E_HIP);
    committed_out[si] = y;
    if (info) info->kstar[si] = kstar;
    s.committed.push_back(y);
    // old anchor's keys/values become committed position A.pos
    J[6 * njobs + 0] = si; J[6 * njobs + 1] = slot_entry(ctx, s, 0); J[6 * njobs + 2] = A.pos;
    J[6 * njobs + 3] = 0; J[6 * njobs + 4] = 0; J[6 * njobs + 5] = 0;
    ++njobs;
    const int child = (kstar <= N - 2) ? A.child[kstar] : -1;
    std::vector<int> keep;
    if (child >= 0) {
      for (int i = 0; i < (int)s.slots.size(); ++i) {
        int t = i;
        while (t >= 0 && t != child) t = s.slots[t].parent;
        if (t == child) keep.push_back(i);
      }
    }
    const int nh = 1 - s.half;
    std::vector<Slot> ns;
    if (!keep.empty()) {
      std::vector<int> remap(s.slots.size(), -1);
      for (int j = 0; j < (int)keep.size(); ++j) remap[keep[j]] = j;
      for (int j = 0; j < (int)keep.size(); ++j) {
        Slot sl = s.slots[keep[j]];
        sl.parent = (keep[j] == child) ? -1 : remap[sl.parent];
        if (keep[j] == child) sl.fork_stage = -1;
        for (int &ch : sl.child) ch = (ch >= 0) ? remap[ch] : -1;
        ns.push_back(sl);
        J[6 * njobs + 0] = si;
        J[6 * njobs + 1] = ctx->max_ctx + s.half * ctx->S + keep[j];
        J[6 * njobs + 2] = ctx->max_ctx + nh * ctx->S + j;
        J[6 * njobs + 3] = s.half * ctx->S + keep[j];
        J[6 * njobs + 4] = nh * ctx->S + j;
        J[6 * njobs + 5] = 1;
        ++njobs;
      }
    } else {
      Slot f;
      f.x = y; f.pos = A.pos + 1; f.child.assign(N, -1);
      ns.push_back(f);
    }
    s.slots = ns;
    s.half = nh;
    s.last_map = keep;
    s.last_fresh = keep.empty() ? 1 : 0;
    s.last_committed_pos = A.pos;
    if ((int)s.committed.size() >= ctx->max_ctx) s.active = false;
  }
  if (njobs > 0) {
    HIPCHK(hipMemcpyAsync(ctx->job_dev, J, njobs * 6 * 4, hipMemcpyHostToDevice, ctx->stream));
    CollapseArgs c{};
    c.n_jobs = njobs; c.job = ctx->job_dev; c.kc = ctx->kc; c.vc = ctx->vc;
    c.n_layers = ctx->L; c.batch = B; c.n_kv_heads = ctx->Hkv; c.kv_entries = ctx->E; c.head_dim = ctx->hd;
    c.elem_bytes = ctx->es; c.bnd_h = ctx->bnd_h; c.bnd_part = ctx->bnd_part; c.cand = ctx->cand;
    c.slots2 = 2 * ctx->S; c.d = ctx->d; c.n_part = ctx->n_part; c.N = N; c.max_ctx = ctx->max_ctx; c.S = ctx->S;
    TimedLaunch tl(ctx, 7, 0.0);
    HIPCHK(launch_collapse(c, ctx->stream));
  }
  if (rt) {
    HIPCHK(hipEventRecord(rt[5], ctx->stream));
    ctx->rt_prev = true;
    ctx->rt_cur = 1 - ctx->rt_cur;
  }
  return DEX_OK;
}

dex_status dex_debug_set_round_timing(dex_ctx *ctx, int32_t enable) {
  if (!ctx) return DEX_E_INVAL;
  for (auto &set : ctx->rt_ev)
    for (auto &e : set)
      if (!e && hipEventCreate(&e) != hipSuccess) { ctx->err = "hipEventCreate failed"; return DEX_E_HIP; }
  ctx->round_timing = enable != 0;
  ctx->rt_prev = false;
  ctx->rt_rounds = 0;
  for (double &v : ctx->rt_ms) v = 0.0;
  return DEX_OK;
}

dex_status dex_debug_round_times(dex_ctx *ctx, int32_t n, double *ms, int64_t *rounds) {
  if (!ctx || !ms || !rounds || n < 0 || n > kRoundPhases) return DEX_E_INVAL;
  for (int i = 0; i < n; ++i) ms[i] = ctx->rt_ms[i];
  *rounds = ctx->rt_rounds;
  return DEX_OK;
}

dex_status dex_debug_plan(int32_t n_explored, int32_t width_cap, int32_t decs, int32_t max_context,
                          const int32_t *slots, int32_t n_slots, int32_t *out, int32_t capacity, int32_t *n_out) {
  const int N = n_explored;
  if (N < 1 || N > DEX_MAX_EXPLORED || width_cap < 0 || max_context < 2 || !slots || n_slots < 1 || !out ||
      !n_out || capacity < 0)
    return DEX_E_INVAL;
  const int st = 4 + N;
  Seq s;
  s.slots.resize(n_slots);
  for (int i = 0; i < n_slots; ++i) {
    const int32_t *r = slots + (size_t)i * st;
    Slot &sl = s.slots[i];
    sl.parent = r[0]; sl.fork_stage = r[1]; sl.c = r[2]; sl.pos = r[3];
    if ((i == 0) != (sl.parent < 0) || sl.parent >= i || sl.c < 0 || sl.c > N) return DEX_E_INVAL;
    if (i > 0 && (sl.fork_stage < 0 || sl.fork_stage >= s.slots[sl.parent].c || sl.fork_stage > N - 2))
      return DEX_E_INVAL;
    sl.u.assign(r + 4, r + 4 + sl.c);
    sl.child.assign(N, -1);
    if (i > 0) {
      Slot &p = s.slots[sl.parent];
      if (p.child[sl.fork_stage] >= 0) return DEX_E_INVAL;
      p.child[sl.fork_stage] = i;
      sl.x = p.u[sl.fork_stage];
    }
  }
  const std::vector<Item> items = plan_items(PlanRule{N, width_cap, decs ? 1 : 0, max_context}, s);
  *n_out = (int)items.size();
  if ((int)items.size() > capacity) return DEX_E_INVAL;
  for (size_t j = 0; j < items.size(); ++j) {
    out[3 * j] = items[j].kind;
    out[3 * j + 1] = items[j].slot;
    out[3 * j + 2] = items[j].f;
  }
  return DEX_OK;
}

dex_status dex_debug_set_logits_tap(dex_ctx *ctx, float *buf, int32_t cap) {
  if (!ctx) return DEX_E_INVAL;
  if (buf && cap < ctx->R_max) { ctx->err = "logits tap capacity below rows per round"; return DEX_E_INVAL; }
  ctx->logits_tap = buf;
  ctx->logits_cap = cap;
  return DEX_OK;
}

dex_status dex_debug_lattice(dex_ctx *ctx, int32_t seq, int32_t *out, int32_t cap, int32_t *n) {
  if (!ctx || !out || !n || seq < 0 || seq >= ctx->B) return DEX_E_INVAL;
  const Seq &s = ctx->seqs[seq];
  *n = (int)s.slots.size();
  if (cap < *n) { ctx->err = "slot table capacity too small"; return DEX_E_INVAL; }
  const int st = 5 + ctx->N;
  for (int i = 0; i < *n; ++i) {
    const Slot &sl = s.slots[i];
    int *o = out + i * st;
    o[0] = sl.x; o[1] = sl.pos; o[2] = sl.parent; o[3] = sl.fork_stage; o[4] = sl.c;
    for (int j = 0; j < ctx->N; ++j) o[5 + j] = j < (int)sl.u.size() ? sl.u[j] : -1;
  }
  return DEX_OK;
}

dex_status dex_debug_last_collapse(dex_ctx *ctx, int32_t seq, int32_t *map, int32_t cap, int32_t *n,
                                   int32_t *fresh, int32_t *cpos) {
  if (!ctx || !map || !n || !fresh || !cpos || seq < 0 || seq >= ctx->B) return DEX_E_INVAL;
  const Seq &s = ctx->seqs[seq];
  *n = (int)s.last_map.size();
  if (cap < *n) return DEX_E_INVAL;
  for (int i = 0; i < *n; ++i) map[i] = s.last_map[i];
  *fresh = s.last_fresh;
  *cpos = s.last_committed_pos;
  return DEX_OK;
}

dex_status dex_debug_kv_layout(dex_ctx *ctx, void **k, void **v, int64_t *entries) {
  if (!ctx || !k || !v || !entries) return DEX_E_INVAL;
  *k = ctx->kc;
  *v = ctx->vc;
  *entries = ctx->E;
  return DEX_OK;
}

dex_status dex_debug_slot_entry(dex_ctx *ctx, int32_t seq, int32_t slot, int32_t *entry) {
  if (!ctx || !entry || seq < 0 || seq >= ctx->B) return DEX_E_INVAL;
  if (slot < 0 || slot >= ctx->S) return DEX_E_INVAL;
  *entry = slot_entry(ctx, ctx->seqs[seq], slot);
  return DEX_OK;
}

dex_status dex_debug_set_kernel_timing(dex_ctx *ctx, int32_t enable) {
  if (!ctx) return DEX_E_INVAL;
  ctx->timing = enable != 0;
  for (int i = 0; i < 8; ++i) { ctx->t_ms[i] = 0; ctx->t_n[i] = 0; ctx->t_bytes[i] = 0; }
  return DEX_OK;
}

dex_status dex_debug_kernel_times(dex_ctx *ctx, int32_t n, double *ms, int64_t *launches, double *bytes) {
  if (!ctx || n < 0 || n > 8) return DEX_E_INVAL;
  for (int i = 0; i < n; ++i) {
    if (ms) ms[i] = ctx->t_ms[i];
    if (launches) launches[i] = ctx->t_n[i];
    if (bytes) bytes[i] = ctx->t_bytes[i];
  }
  return DEX_OK;
}

dex_status dex_debug_time_kernel(dex_ctx *ctx, int32_t cls, int32_t M, int32_t reps, double *avg_us,
                                 double *bytes_per_launch) {
  if (!ctx || !avg_us || !bytes_per_launch || M < 1 || M > ctx->R_max || reps < 1) return DEX_E_INVAL;
  if (cls != 3 && cls != 4 && cls != 5 && cls != 6) { ctx->err = "only o-proj, gate/up, down, lm-head"; return DEX_E_INVAL; }
  if (!ctx->prefilled) { ctx->err = "time_kernel needs a prefilled context"; return DEX_E_STATE; }
  const int d = ctx->d, H = ctx->H, hd = ctx->hd, F = ctx->F;
  struct Events {
    hipEvent_t e0 = nullptr, e1 = nullptr;
    ~Events() {
      if (e0) (void)hipEventDestroy(e0);
      if (e1) (void)hipEventDestroy(e1);
    }
  } ev;
  HIPCHK(hipEventCreate(&ev.e0));
  HIPCHK(hipEventCreate(&ev.e1));
  hipEvent_t e0 = ev.e0, e1 = ev.e1;
  double bytes = 0.0;
  auto launch = [&](int rep) -> hipError_t {
    const int l = rep % ctx->L;
    GemmArgs a{};
    a.M = M;
    int epi = EPI_RESID;
    if (cls == 3) {
      a.wp = ctx->p_o[l]; a.nsteps_w = ctx->ns_hhd; a.N = d; a.K = H * hd; a.x = ctx->att_w; a.ldx = H * hd;
      a.h = ctx->h_w; a.ld_h = d; a.alpha = 0.f; a.part_out = ctx->part_w; a.n_part_out = ctx->n_part;
      bytes = (double)ctx->es * ((double)d * H * hd + (double)M * H * hd + (double)M * d) + 8.0 * M * d;
    } else if (cls == 4) {
      a.wp = ctx->p_gu[l]; a.nsteps_w = ctx->ns_d; a.N = F; a.K = d; a.x = ctx->xb_w; a.ldx = d;
      a.part = ctx->part_w; a.n_part = ctx->n_part; a.inv_d = 1.0f / d; a.eps = ctx->eps;
      a.act = ctx->act_w; a.ld_act = F;
      epi = EPI_SWIGLU;
      bytes = (double)ctx->es * (2.0 * F * d + (double)M * d + (double)M * F);
    } else if (cls == 5) {
      a.wp = ctx->p_down[l]; a.nsteps_w = ctx->ns_F; a.N = d; a.K = F; a.x = ctx->act_w; a.ldx = F;
      a.h = ctx->h_w; a.ld_h = d; a.alpha = 0.f; a.part_out = ctx->part_w; a.n_part_out = ctx->n_part;
      bytes = (double)ctx->es * ((double)d * F + (double)M * F + (double)M * d) + 8.0 * M * d;
    } else {
      a.wp = ctx->p_lm; a.nsteps_w = ctx->ns_d; a.N = ctx->V; a.K = d; a.x = ctx->ex_xb; a.ldx = d;
      a.part = ctx->ex_part; a.n_part = ctx->n_part; a.inv_d = 1.0f / d; a.eps = ctx->eps;
      a.mask_n = ctx->tab_dev; a.mask_tok = ctx->tab_dev; a.mask_stride = 0;
      a.amax = ctx->amax; a.n_tiles = (ctx->V + 15) / 16;
      epi = EPI_LOGITS;
      bytes = (double)ctx->es * ((double)ctx->V * d + (double)M * d);
    }
    return launch_gemm(ctx->dtype, epi, a, 1, ctx->stream);
  };
  // zero mask counts for the LM head (the row tables are rewritten every round)
  if (cls == 6) HIPCHK(hipMemsetAsync(ctx->tab_dev, 0, (size_t)M * 4, ctx->stream));
  HIPCHK(launch(0));                       // warm the code object
  HIPCHK(hipEventRecord(e0, ctx->stream));
  for (int i = 0; i < reps; ++i) HIPCHK(launch(i + 1));
  HIPCHK(hipEventRecord(e1, ctx->stream));
  HIPCHK(hipEventSynchronize(e1));
  float ms = 0.f;
  HIPCHK(hipEventElapsedTime(&ms, e0, e1));
  *avg_us = (double)ms * 1e3 / reps;
  *bytes_per_launch = bytes;
  return DEX_OK;
}

dex_status dex_debug_gemm(int32_t dtype, const void *W, int32_t N, int32_t K, const void *x, int32_t M, float *y,
                          void *stream) {
  if (!W || !x || !y || N < 1 || K < 1 || M < 1) return DEX_E_INVAL;
  if (dtype != DEX_F32 && dtype != DEX_BF16) return DEX_E_INVAL;
  if (M > 64 && (dtype != DEX_BF16 || N % 16)) return DEX_E_INVAL;
  if (K % (dtype == DEX_BF16 ? 8 : 4)) return DEX_E_INVAL;
  void *wp = nullptr;
  if (hipMalloc(&wp, packed_bytes(dtype, N, K, 0)) != hipSuccess) return DEX_E_NOMEM;
  PackArgs pa{};
  pa.w0 = W; pa.n0 = N; pa.N = N; pa.K = K; pa.mode = 0; pa.head_dim = 16; pa.out = wp;
  hipError_t e = launch_pack(dtype, pa, (hipStream_t)stream);
  GemmArgs a{};
  a.wp = wp; a.nsteps_w = (K + (dtype == DEX_BF16 ? 32 : 16) - 1) / (dtype == DEX_BF16 ? 32 : 16);
  a.N = N; a.K = K; a.x = x; a.ldx = K; a.M = M; a.out = y; a.ld_out = N;
  if (e == hipSuccess)
    e = M > 64 ? launch_gemm_tiled(EPI_PLAIN, a, (hipStream_t)stream) : launch_gemm(dtype, EPI_PLAIN, a, 1, (hipStream_t)stream);
  if (e == hipSuccess) e = hipStreamSynchronize((hipStream_t)stream);
  (void)hipFree(wp);
  return e == hipSuccess ? DEX_OK : DEX_E_HIP;
}

dex_status dex_debug_attention(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                               int32_t batch, int32_t kv_entries, const void *k_cache, const void *v_cache,
                               const float *q, int32_t n_rows, const int32_t *row_seq, const int32_t *row_pos,
                               const int32_t *row_nc, const int32_t *chain_off, const int32_t *chain,
                               int32_t chain_len, void *out, void *stream) {
  const AttnCall c{dtype, head_dim, n_heads, n_kv_heads, batch, kv_entries, k_cache, v_cache, q, n_rows,
                   row_seq, row_pos, row_nc, chain_off, chain, chain_len, out};
  if (n_rows < 1 || chain_len < 0) return DEX_E_INVAL;
  std::vector<int> tab(attention_table_ints(n_rows, chain_len));
  AttnTab t{};
  const dex_status vs = attention_tables(c, tab.data(), tab.size(), &t);
  if (vs != DEX_OK) return vs;
  const hipStream_t st = (hipStream_t)stream;
  int *dtab = nullptr;
  float *part = nullptr;
  if (hipMalloc((void **)&dtab, t.n_ints * 4) != hipSuccess) return DEX_E_NOMEM;
  if (hipMalloc((void **)&part, t.part_bytes) != hipSuccess) { (void)hipFree(dtab); return DEX_E_NOMEM; }
  hipError_t e = hipMemcpyAsync(dtab, tab.data(), t.n_ints * 4, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = launch_attention_call(c, t, dtab, part, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  else (void)hipStreamSynchronize(st);
  (void)hipFree(part);
  (void)hipFree(dtab);
  return e == hipSuccess ? DEX_OK : DEX_E_HIP;
}

dex_status dex_debug_attention_noalloc(int32_t dtype, int32_t head_dim, int32_t n_heads, int32_t n_kv_heads,
                                       int32_t batch, int32_t kv_entries, const void *k_cache,
                                       const void *v_cache, const float *q, int32_t n_rows,
                                       const int32_t *row_seq, const int32_t *row_pos, const int32_t *row_nc,
                                       const int32_t *chain_off, const int32_t *chain, int32_t chain_len,
                                       void *out, void *stream) {
  g_create_error.clear();
  const AttnCall c{dtype, head_dim, n_heads, n_kv_heads, batch, kv_entries, k_cache, v_cache, q, n_rows,
                   row_seq, row_pos, row_nc, chain_off, chain, chain_len, out};
  if (n_rows < 1 || chain_len < 0) return DEX_E_INVAL;
  if (n_rows > DEX_MAX_ROWS || chain_len > kNoallocMaxChain) {
    g_create_error = "dex_debug_attention_noalloc: more than 256 rows or 16384 chain entries";
    return DEX_E_CAPACITY;
  }
  // host staging of the tables: a fixed per-thread array (no allocation)
  thread_local int tab[kNoallocTableInts];
  AttnTab t{};
  const dex_status vs = attention_tables(c, tab, kNoallocTableInts, &t);
  if (vs != DEX_OK) return vs;
  if (t.part_bytes > kScratchBytes - kScratchTableBytes) {
    g_create_error = "dex_debug_attention_noalloc: split partials exceed the 63.75 MiB scratch";
    return DEX_E_CAPACITY;
  }
  void *base = nullptr;
  hipError_t e = scratch_address(&base);
  if (e != hipSuccess) {
    g_create_error = std::string("scratch address: ") + hipGetErrorString(e);
    return DEX_E_HIP;
  }
  const hipStream_t st = (hipStream_t)stream;
  int *dtab = (int *)base;
  float *part = (float *)((char *)base + kScratchTableBytes);
  e = hipMemcpyAsync(dtab, tab, t.n_ints * 4, hipMemcpyHostToDevice, st);
  if (e == hipSuccess) e = launch_attention_call(c, t, dtab, part, st);
  if (e == hipSuccess) e = hipStreamSynchronize(st);
  else (void)hipStreamSynchronize(st);
  return e == hipSuccess ? DEX_OK : DEX_E_HIP;
}

dex_status dex_debug_gumbel(uint64_t seed, int32_t seq, int32_t pos, int32_t V, float *out, void *stream) {
  if (!out || V < 1 || seq < 0 || pos < 0) return DEX_E_INVAL;
  hipError_t e = launch_gumbel(seed, seq, pos, V, out, (hipStream_t)stream);
  return e == hipSuccess ? DEX_OK : DEX_E_HIP;
}

dex_status dex_debug_copy(void *dst, const void *src, int64_t bytes, void *stream) {
  if (!dst || !src || bytes < 0 || bytes % 16) return DEX_E_INVAL;
  hipError_t e = launch_copy(dst, src, bytes, (hipStream_t)stream);
  return e == hipSuccess ? DEX_OK : DEX_E_HIP;
}

}  // extern "C"
