// Host side of the C ABI: argument checks, workspace carving, tables, and the launch sequence of
// prefill and of one pipeline step on the caller's two streams.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <new>
#include <random>
#include <string>
#include <vector>

#include "spd.h"
#include "spd_dev.h"

using namespace spd;

namespace {

thread_local std::string g_init_error;

enum HState { H_INIT = 0, H_READY = 1, H_PENDING = 2 };

struct Layout {
  size_t kv, pkv, pt, rope, state, tok, forced, log, resid, anch, pdmx, pfx, pfanch, dbg, lay;
  size_t q[2], ao[2], act[2], part[2], cnt[2], hkey[2], rpart[2], rtick[2];
  size_t ktrace;
  size_t su, swlog, swgmax, sqids, sqp, sqcnt, spq;  // sampled decoding
  size_t total;
  int wlog_stride;
  int num_pages, chunk, max_splits, J, nkslots;
  size_t kv_layer_bytes;
};

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

spd_status check_config(const spd_config* c, std::string* why) {
  auto bad = [&](const char* m) {
    if (why) *why = m;
    return SPD_E_INVAL;
  };
  if (!c) return bad("config is NULL");
  if (c->n_layers < 1 || c->d_model < 8 || c->n_q_heads < 1 || c->n_kv_heads < 1 || c->ffn_dim < 8 ||
      c->vocab < 1)
    return bad("dimensions must be positive");
  if (c->head_dim != 64 && c->head_dim != 128) return bad("head_dim must be 64 or 128");
  if (c->n_q_heads % c->n_kv_heads) return bad("n_q_heads must be a multiple of n_kv_heads");
  const int G = c->n_q_heads / c->n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return bad("n_q_heads / n_kv_heads must be 1, 2, 4 or 8");
  if (c->d_model % 8 || c->ffn_dim % 8 || (c->n_q_heads * c->head_dim) % 8)
    return bad("d_model, ffn_dim and n_q_heads*head_dim must be multiples of 8");
  if (c->dtype != SPD_F32 && c->dtype != SPD_BF16) return bad("dtype must be SPD_F32 or SPD_BF16");
  if (c->n_stages < 1 || c->n_stages > kMaxStages || c->n_stages > c->n_layers)
    return bad("n_stages must be in [1, min(8, n_layers)]");
  if (c->pdm_layers < 1 || c->pdm_layers > kMaxPdmLayers) return bad("pdm_layers must be in [1, 4]");
  if (c->page_size != 16) return bad("page_size must be 16");
  if (c->max_tokens < c->n_stages + 2) return bad("max_tokens too small");
  if (c->max_tokens > (1 << 20)) return bad("max_tokens too large");
  if (c->attn_chunk < 0 || (c->attn_chunk && (c->attn_chunk % c->page_size)))
    return bad("attn_chunk must be 0 or a multiple of page_size");
  if (c->attn_chunk && (c->max_tokens + c->attn_chunk - 1) / c->attn_chunk > kMaxSplits)
    return bad("attn_chunk too small: max_tokens / attn_chunk must not exceed 64 key splits");
  if (!(c->rms_eps > 0.f) || !(c->rope_base > 1.f)) return bad("rms_eps must be > 0 and rope_base > 1");
  if (c->auto_rollback != 0 && c->auto_rollback != 1) return bad("auto_rollback must be 0 or 1");
  if (c->fused_head != 0 && c->fused_head != 1) return bad("fused_head must be 0 or 1");
  if (c->pdm_vocab < 0 || c->pdm_vocab > c->vocab) return bad("pdm_vocab must be in [0, vocab]");
  if (c->pdm_vocab > 0 && c->fused_head) return bad("an own PDM head (pdm_vocab > 0) needs fused_head = 0");
  if (c->d_model > 8192) return bad("d_model must be at most 8192");
  return SPD_OK;
}

// Floats of one set's K-split row GEMV records: the largest sublayer's chunk dot products (chunks x
// kMaxRows rows x pairs x 2), then the sums of squares of up to kRowSplitCols columns.
size_t rows_split_floats(const spd_config& c) {
  const int d = c.d_model, qdim = c.n_q_heads * c.head_dim, F = c.ffn_dim;
  auto chunks = [](int K) { return (size_t)(K + kRowSplitK - 1) / kRowSplitK; };
  const size_t pairs_qkv = (size_t)(c.n_q_heads + 2 * c.n_kv_heads) * (c.head_dim / 2);
  const size_t pairs_half = (size_t)(d + 1) / 2;
  size_t rec = chunks(d) * pairs_qkv;
  rec = std::max(rec, chunks(qdim) * pairs_half);
  rec = std::max(rec, chunks(d) * (size_t)F);
  rec = std::max(rec, chunks(F) * pairs_half);
  const size_t max_chunks = std::max(chunks(d), std::max(chunks(qdim), chunks(F)));
  return rec * kMaxRows * 2 + (size_t)kRowSplitCols * max_chunks * kMaxRows;
}

Layout make_layout(const spd_config& c) {
  Layout L{};
  const size_t esz = c.dtype == SPD_BF16 ? 2 : 4;
  const int n = c.n_stages, d = c.d_model, dh = c.head_dim, hkv = c.n_kv_heads;
  const int qdim = c.n_q_heads * dh;
  const int G = c.n_q_heads / hkv;
  L.num_pages = (c.max_tokens + c.page_size - 1) / c.page_size;
  // about 40 key splits at full capacity, at least 64 keys each: enough workgroups for the short
  // contexts, few partials for the long ones (never more than kMaxSplits)
  {
    const int ch = ((c.max_tokens + 39) / 40 + 63) / 64 * 64;
    L.chunk = c.attn_chunk ? c.attn_chunk : std::max(64, ch);
  }
  L.max_splits = (c.max_tokens + L.chunk - 1) / L.chunk;
  // layer slots per step: the longest stage
  L.J = 0;
  for (int s = 0; s < n; s++)
    L.J = std::max(L.J, (int)((long long)(s + 1) * c.n_layers / n) - (int)((long long)s * c.n_layers / n));
  L.kv_layer_bytes = (size_t)L.num_pages * 2 * hkv * c.page_size * dh * esz;
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  L.kv = take(L.kv_layer_bytes * c.n_layers);
  L.pkv = take(L.kv_layer_bytes * c.pdm_layers);
  L.pt = take(sizeof(int32_t) * L.num_pages);
  L.rope = take(sizeof(float) * 2 * (size_t)c.max_tokens * (dh / 2));
  L.state = take(sizeof(DevState));
  L.tok = take(sizeof(int32_t) * (c.max_tokens + 8));
  L.forced = take(sizeof(int32_t) * (c.max_tokens + 8));
  L.log = take(sizeof(spd_step_result) * kLogCap);
  L.resid = take(sizeof(float) * n * d);
  L.anch = take(sizeof(float) * n * n * d);
  L.pdmx = take(sizeof(float) * kMaxRows * d);
  L.pfx = take(sizeof(float) * kMaxRows * d);
  L.pfanch = take(sizeof(float) * kMaxRows * n * d);
  L.dbg = take(sizeof(float) * 2 * (size_t)c.vocab);
  L.lay = take(sizeof(LayerDesc) * (c.n_layers + c.pdm_layers));
  const size_t part_floats = (size_t)64 * hkv * L.max_splits * (dh + 2);
  (void)G;
  for (int s = 0; s < 2; s++) {
    L.q[s] = take(sizeof(float) * kMaxRows * qdim);
    L.ao[s] = take(sizeof(float) * kMaxRows * qdim);
    L.act[s] = take(sizeof(float) * kMaxRows * (size_t)c.ffn_dim);
    L.part[s] = take(sizeof(float) * part_floats);
    L.cnt[s] = take(sizeof(int32_t) * kMaxStages * hkv);
    L.rpart[s] = take(sizeof(float) * rows_split_floats(c));
    L.rtick[s] = take(sizeof(int32_t) * kRowSplitCols);
    L.hkey[s] = take(sizeof(unsigned long long));
  }
  L.nkslots = 5 * L.J * n + 4;
  L.ktrace = take(sizeof(unsigned long long) * 2 * (size_t)L.nkslots);
  // sampled decoding: the head's wave regions cover at most V + 2 * (4 * kSampleWGs) floats per row
  L.wlog_stride = (int)align_up((size_t)c.vocab + 8 * kSampleWGs, 64);
  L.su = take(sizeof(float) * 3 * (size_t)c.max_tokens);
  L.swlog = take(sizeof(float) * 2 * (size_t)L.wlog_stride);
  L.swgmax = take(sizeof(unsigned long long) * 2 * kSampleWGs);
  L.sqids = take(sizeof(int32_t) * n * kMaxTopK);
  L.sqp = take(sizeof(float) * n * kMaxTopK);
  L.sqcnt = take(sizeof(int32_t) * n);
  L.spq = take((sizeof(int32_t) + sizeof(float)) * kMaxTopK + sizeof(int32_t));
  L.total = o;
  return L;
}

void stage_bounds(int L, int n, int* beta) {
  for (int s = 0; s <= n; s++) beta[s] = (int)((long long)s * L / n);
}

}  // namespace

namespace spd {
// The message spd_last_error(NULL) returns, for calls that have no handle.
void set_call_error(const std::string& msg) { g_init_error = msg; }
}  // namespace spd

struct spd_handle {
  spd_config cfg;
  Layout lay;
  Ctx ctx;
  int dev = 0;
  int bf16 = 0;
  int J = 0;  // layer slots per step = longest stage
  hipStream_t main = nullptr, pdm = nullptr;
  hipEvent_t ev_fork = nullptr, ev_join = nullptr;
  // stage groups (step-kernel mode 2): one stream and one completion event per group (default priority)
  hipStream_t sst[kMaxStages] = {};
  hipEvent_t ev_st[kMaxStages] = {};
  char* ws = nullptr;
  int hstate = H_INIT;
  int c = 0, a = 0, prompt_len = 0;
  int unsynced = 0;     // steps were enqueued since the host last read c and a
  long long bound = 0;  // upper bound of c + a (each step raises c + a by at most one)
  spd_step_result* pinned = nullptr;  // [kLogCap + 1]
  std::vector<int32_t> page_table;
  std::vector<LayerDesc> layer_desc;  // host copy of the layer table
  std::string err;
  // step graph (fork/join of both streams captured once, replayed per step)
  int use_graph = 0;
  // stage compute: 0 = five launches per layer slot on main_stream, 2 = stage groups on their own
  // streams
  int step_mode = 2;
  int stage_groups = 0;  // mode 2: streams the stages are spread over (0: kStageGroupsDefault)
  int pdm_place = 0;     // where the PDM's launches go (spd_set_pdm_placement)
  int pdm_on = 1;        // 0: the step skips the PDM's launches (spd_set_pdm_enabled)
  hipGraphExec_t gexec = nullptr;
  hipGraphExec_t gexec_multi = nullptr;  // graph_steps steps in one graph (spd_run_steps)
  int graph_steps = 1;
  // kernel timing
  int timed_kernel = 0;
  int timed_first_slot = 0;
  int cur_slot = 0;  // layer slot being enqueued (J for the exit head)
  std::vector<hipEvent_t> tev;  // pool, pairs
  size_t tev_used = 0;
  std::vector<hipEvent_t> sev;  // span events, triples (start, pdm end, stage end)
  size_t sev_used = 0;
};

#define HIPC(expr)                                                              \
  do {                                                                          \
    hipError_t e_ = (expr);                                                     \
    if (e_ != hipSuccess) {                                                     \
      h->err = std::string(#expr) + ": " + hipGetErrorString(e_);               \
      return SPD_E_HIP;                                                         \
    }                                                                           \
  } while (0)

static spd_status launch_check(spd_handle* h, const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    h->err = std::string("launch ") + what + ": " + hipGetErrorString(e);
    return SPD_E_HIP;
  }
  return SPD_OK;
}

// Kernel timing of one launch when that launch class is being timed (main stream only): the launch
// inside the scope hands an event pair to its dispatch, which records the kernel's own start and end.
struct TimedLaunch {
  bool on;
  TimedLaunch(spd_handle* h, hipStream_t s, int kind) : on(false) {
    if (!h || h->timed_kernel != kind || h->cur_slot < h->timed_first_slot) return;
    bool ours = s == h->main;
    for (int st = 0; st < kMaxStages; st++) ours = ours || (h->sst[st] != nullptr && s == h->sst[st]);
    if (!ours) return;
    if (h->tev_used + 2 > h->tev.size()) {
      for (int i = 0; i < 64; i++) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return;
        h->tev.push_back(e);
      }
    }
    const size_t idx = h->tev_used;
    h->tev_used += 2;
    set_launch_events(h->tev[idx], h->tev[idx + 1]);
    on = true;
  }
  ~TimedLaunch() {
    if (on) set_launch_events(nullptr, nullptr);
  }
};

template <typename WT>
static void enqueue_layer(const Ctx& C, const Rows& r, hipStream_t s, spd_handle* h = nullptr) {
  { TimedLaunch t(h, s, SPD_K_QKV); Launch<WT>::qkv(C, r, s); }
  { TimedLaunch t(h, s, SPD_K_ATTN); Launch<WT>::attn(C, r, s); }
  { TimedLaunch t(h, s, SPD_K_OPROJ); Launch<WT>::oproj(C, r, s); }
  { TimedLaunch t(h, s, SPD_K_GATEUP); Launch<WT>::gateup(C, r, s); }
  { TimedLaunch t(h, s, SPD_K_DOWN); Launch<WT>::down(C, r, s); }
}

// PDM GEMV workgroups: kRowsWGsDefault per 256 MB of PDM weights (feature projection and decoder
// layers), so that a larger draft module keeps finishing inside the stage compute.
static int default_rows_wgs(const spd_config& c) {
  const double esz = c.dtype == SPD_BF16 ? 2.0 : 4.0;
  const double d = c.d_model, qd = (double)c.n_q_heads * c.head_dim, kvd = (double)c.n_kv_heads * c.head_dim;
  const double layer = d * (qd + 2 * kvd) + qd * d + 3 * d * c.ffn_dim;
  const double bytes = esz * (d * c.n_stages * d + c.pdm_layers * layer);
  const int units = std::max(1, (int)std::lround(bytes / (256.0 * 1024 * 1024)));
  return std::min(kRowsWGsDefault * units, 1024);
}

static Rows rows_block(int layer, int nrows, int pos0, float* x, float* anch, int cap, int set) {
  Rows r;
  std::memset(&r, 0, sizeof(Rows));
  r.kind = 1;
  r.slot = 0;
  r.layer = layer;
  r.nrows = nrows;
  r.pos0 = pos0;
  r.x = x;
  r.anch = anch;
  r.cap = cap;
  r.set = set;
  return r;
}

// Three timing events of one step when SPD_K_SPANS timing is on (nullptr otherwise).
static hipEvent_t* span_events(spd_handle* h) {
  if (h->timed_kernel != SPD_K_SPANS) return nullptr;
  if (h->sev_used + 3 > h->sev.size()) {
    for (int i = 0; i < 96; i++) {
      hipEvent_t e;
      if (hipEventCreate(&e) != hipSuccess) return nullptr;
      h->sev.push_back(e);
    }
  }
  hipEvent_t* ev = h->sev.data() + h->sev_used;
  h->sev_used += 3;
  return ev;
}

template <typename WT>
static spd_status enqueue_step(spd_handle* h, int forced_override) {
  const Ctx& C = h->ctx;
  hipEvent_t* sp = span_events(h);
  if (C.ktrace) launch_ktrace_reset(C, h->lay.nkslots, h->main);
  if (sp) HIPC(hipEventRecord(sp[0], h->main));
  const bool fused = h->cfg.fused_head != 0;
  // Pipeline Draft Module: pre-step features only (Section 3.3), so it can run beside the stage
  // compute; it ends by recording ev_join, which the LM head waits for. Its launches, in order: the
  // feature projection, five per PDM layer, the draft head if not fused.
  auto enqueue_pdm = [&](hipStream_t s) -> spd_status {
    h->cur_slot = 0;
    Launch<WT>::pdm_fc(C, 0, 0, s);
    for (int l = 0; l < h->cfg.pdm_layers; l++)
      Launch<WT>::rows_layer(C, rows_block(h->cfg.n_layers + l, -1, -1, C.pdm_x, nullptr, -1, 1),
                             h->cfg.n_stages, C.rows_wgs, s);
    if (!fused) {
      if (C.sam.top_k > 0)  // the draft module's distribution, left for the exit row's pass
        Launch<WT>::head_sample(C, 1, 0, 0, -1, 0, s);
      else
        Launch<WT>::head(C, 1, 0, s);
    }
    if (sp) HIPC(hipEventRecord(sp[1], s));
    HIPC(hipEventRecord(h->ev_join, s));
    return SPD_OK;
  };
  const bool stage_streams = h->step_mode == 2;
  // post-step schedule: the PDM waits for the stage compute (placement 5, on main_stream after it)
  const int place = !h->pdm_on ? -1 : C.post_step ? 5 : stage_streams ? h->pdm_place : (h->pdm_place == 1 ? 1 : 0);
  if (place == -1) {  // no PDM launches: the join is satisfied at the fork
    if (sp) HIPC(hipEventRecord(sp[1], h->main));
    HIPC(hipEventRecord(h->ev_join, h->main));
  }
  if (place == 1) {  // on main_stream, before the stage compute
    spd_status st = enqueue_pdm(h->main);
    if (st != SPD_OK) return st;
  }
  HIPC(hipEventRecord(h->ev_fork, h->main));
  if (place == 0) {  // its own stream
    HIPC(hipStreamWaitEvent(h->pdm, h->ev_fork, 0));
    spd_status st = enqueue_pdm(h->pdm);
    if (st != SPD_OK) return st;
  }
  // every active stage advances its token by one layer per slot (Section 3.1). mode 0: every launch
  // covers all stages, on main_stream. mode 2: the stages are spread over G groups of consecutive
  // stages, each group running its own chain of launches (covering its stages) on its own stream,
  // forked from and joined to main_stream, so that one group's latency-bound attention and launch
  // tails overlap the other groups' weight streaming.
  const int n = h->cfg.n_stages;
  const int groups =
      h->step_mode == 2 ? std::min(h->stage_groups > 0 ? h->stage_groups : kStageGroupsDefault, n) : 1;
  hipStream_t gs[kMaxStages];
  for (int gi = 0; gi < groups; gi++) {
    gs[gi] = h->step_mode == 2 ? h->sst[gi] : h->main;
    if (h->step_mode == 2) HIPC(hipStreamWaitEvent(gs[gi], h->ev_fork, 0));
  }
  if (place == 2) {  // first group's stream, before its stage launches
    spd_status st = enqueue_pdm(gs[0]);
    if (st != SPD_OK) return st;
  }
  for (int j = 0; j < h->J; j++) {
    for (int gi = 0; gi < groups; gi++) {
      const int s0 = gi * n / groups, s1 = (gi + 1) * n / groups;
      h->cur_slot = j;
      Rows r;
      std::memset(&r, 0, sizeof(Rows));
      r.kind = 0;
      r.slot = j;
      r.stage0 = s0;
      r.nst = s1 - s0;
      r.nrows = 1;
      r.cap = -1;
      bool any = false;
      for (int st = 0; st < kMaxStages; st++) {
        const int l = (st >= r.stage0 && st < r.stage0 + r.nst) ? C.beta[st] + j : -1;
        if (l >= 0 && l < C.beta[st + 1]) {
          r.ld[st] = h->layer_desc[l];
          any = true;
        } else {
          std::memset(&r.ld[st], 0, sizeof(LayerDesc));
        }
      }
      if (any) enqueue_layer<WT>(C, r, gs[gi], h);
    }
  }
  if (place == 3) {  // first group's stream, after its stage launches
    spd_status st = enqueue_pdm(gs[0]);
    if (st != SPD_OK) return st;
  }
  if (h->step_mode == 2) {
    for (int gi = 0; gi < groups; gi++) {
      HIPC(hipEventRecord(h->ev_st[gi], gs[gi]));
      HIPC(hipStreamWaitEvent(h->main, h->ev_st[gi], 0));
    }
  }
  if (place == 5) {  // post-step features: after every stage of this step, before the exit head
    h->cur_slot = 0;
    spd_status st = enqueue_pdm(h->main);
    if (st != SPD_OK) return st;
  }
  h->cur_slot = h->J;
  if (fused) {
    // one pass over the vocabulary for the exit row and the draft module's last row
    if (sp) HIPC(hipEventRecord(sp[2], h->main));
    HIPC(hipStreamWaitEvent(h->main, h->ev_join, 0));
    TimedLaunch t(h, h->main, SPD_K_HEAD);
    if (C.sam.top_k > 0)  // + top-k distributions, the draft's draw and the rejection-sampling verify
      Launch<WT>::head_sample(C, 3, 0, 0, forced_override, h->cfg.auto_rollback, h->main);
    else
      Launch<WT>::head_verify(C, 1, forced_override, h->cfg.auto_rollback, h->main);  // + the step's verify
    return launch_check(h, "step");
  }
  // the draft module's own head pass has left its draft: the exit row alone, with the verify in the
  // launch's last workgroup (the draft module ends well inside the stage compute)
  if (sp) HIPC(hipEventRecord(sp[2], h->main));
  HIPC(hipStreamWaitEvent(h->main, h->ev_join, 0));
  TimedLaunch t(h, h->main, SPD_K_HEAD);
  if (C.sam.top_k > 0)  // + the exit row's distribution, the draft's draw and the sampled verify
    Launch<WT>::head_sample(C, 0, 0, 0, forced_override, h->cfg.auto_rollback, h->main);
  else
    Launch<WT>::head_verify(C, 0, forced_override, h->cfg.auto_rollback, h->main);
  return launch_check(h, "step");
}

template <typename WT>
static spd_status enqueue_prefill(spd_handle* h, int len) {
  const Ctx& C = h->ctx;
  const int n = h->cfg.n_stages, L = h->cfg.n_layers;
  for (int t0 = 0; t0 < len; t0 += kMaxRows) {
    const int rc = std::min(kMaxRows, len - t0);
    Launch<WT>::embed_rows(C, t0, rc, h->main);
    for (int l = 0; l < L; l++) {
      int cap = -1;
      for (int s = 0; s + 1 <= n - 1; s++)
        if (l + 1 == C.beta[s + 1]) cap = s + 1;
      Launch<WT>::rows_layer(C, rows_block(l, rc, t0, C.pf_x, C.pf_anch, cap, 0), kMaxRows, 0, h->main);
    }
    // PDM KV over the prompt: every prompt row has full depth
    Launch<WT>::pdm_fc(C, 1, rc, h->main);
    for (int i = 0; i < h->cfg.pdm_layers; i++)
      Launch<WT>::rows_layer(C, rows_block(L + i, rc, t0, C.pdm_x, nullptr, -1, 1), kMaxRows, 0, h->main);
    if (t0 + rc == len) {
      if (C.sam.top_k > 0)  // the first token is drawn from the top-k distribution
        Launch<WT>::head_sample(C, 2, rc - 1, len, -1, 0, h->main);
      else
        Launch<WT>::head(C, 2, rc - 1, h->main);
    }
    spd_status st = launch_check(h, "prefill");
    if (st != SPD_OK) return st;
  }
  launch_reseed(C, len, -1, len, h->main, h->bf16);
  return launch_check(h, "prefill reseed");
}

extern "C" {

const char* spd_status_str(spd_status s) {
  switch (s) {
    case SPD_OK: return "SPD_OK";
    case SPD_E_INVAL: return "SPD_E_INVAL: invalid argument";
    case SPD_E_STATE: return "SPD_E_STATE: call not legal in this state";
    case SPD_E_CAPACITY: return "SPD_E_CAPACITY: capacity exceeded";
    case SPD_E_HIP: return "SPD_E_HIP: HIP runtime error";
  }
  return "unknown spd_status";
}

const char* spd_last_error(const spd_handle* h) { return h ? h->err.c_str() : g_init_error.c_str(); }

spd_status spd_workspace_size(const spd_config* cfg, size_t* bytes) {
  if (!bytes) return SPD_E_INVAL;
  spd_status st = check_config(cfg, &g_init_error);
  if (st != SPD_OK) return st;
  *bytes = make_layout(*cfg).total;
  return SPD_OK;
}

spd_status spd_stage_bounds(const spd_config* cfg, int32_t* beta) {
  if (!beta) return SPD_E_INVAL;
  spd_status st = check_config(cfg, &g_init_error);
  if (st != SPD_OK) return st;
  stage_bounds(cfg->n_layers, cfg->n_stages, beta);
  return SPD_OK;
}

static bool layer_ok(const spd_layer_weights& l) {
  return l.attn_norm && l.wq && l.wk && l.wv && l.wo && l.mlp_norm && l.wg && l.wu && l.wd;
}

spd_status spd_init(const spd_config* cfg, const spd_weights* w, void* workspace, size_t ws_bytes,
                    void* main_stream, void* pdm_stream, spd_handle** out) {
  g_init_error.clear();
  if (!out) return SPD_E_INVAL;
  *out = nullptr;
  spd_status st = check_config(cfg, &g_init_error);
  if (st != SPD_OK) return st;
  if (!w || !w->embed || !w->layers || !w->final_norm || !w->lm_head || !w->pdm_in || !w->pdm_layers ||
      !w->pdm_norm) {
    g_init_error = "weights: NULL pointer";
    return SPD_E_INVAL;
  }
  if (cfg->pdm_vocab > 0 && (!w->pdm_lm_head || !w->pdm_vocab_map)) {
    g_init_error = "weights: pdm_vocab > 0 needs pdm_lm_head and pdm_vocab_map";
    return SPD_E_INVAL;
  }
  for (int l = 0; l < cfg->n_layers; l++)
    if (!layer_ok(w->layers[l])) {
      g_init_error = "weights: NULL layer pointer";
      return SPD_E_INVAL;
    }
  for (int l = 0; l < cfg->pdm_layers; l++)
    if (!layer_ok(w->pdm_layers[l])) {
      g_init_error = "weights: NULL PDM layer pointer";
      return SPD_E_INVAL;
    }
  if (!workspace || ((uintptr_t)workspace & 255)) {
    g_init_error = "workspace must be non-NULL and 256-byte aligned";
    return SPD_E_INVAL;
  }
  if (!main_stream || !pdm_stream || main_stream == pdm_stream) {
    g_init_error = "main_stream and pdm_stream must be two distinct non-default streams";
    return SPD_E_INVAL;
  }
  const Layout lay = make_layout(*cfg);
  if (ws_bytes < lay.total) {
    g_init_error = "workspace too small";
    return SPD_E_CAPACITY;
  }
  spd_handle* h = new (std::nothrow) spd_handle();
  if (!h) return SPD_E_CAPACITY;
  h->cfg = *cfg;
  h->lay = lay;
  h->bf16 = cfg->dtype == SPD_BF16;
  h->main = (hipStream_t)main_stream;
  h->pdm = (hipStream_t)pdm_stream;
  h->ws = (char*)workspace;
  auto fail = [&](spd_status s) {
    g_init_error = h->err;
    spd_destroy(h);
    return s;
  };
#define HIPI(expr)                                                  \
  do {                                                              \
    hipError_t e_ = (expr);                                         \
    if (e_ != hipSuccess) {                                         \
      h->err = std::string(#expr) + ": " + hipGetErrorString(e_);   \
      return fail(SPD_E_HIP);                                       \
    }                                                               \
  } while (0)
  HIPI(hipGetDevice(&h->dev));
  HIPI(hipEventCreateWithFlags(&h->ev_fork, hipEventDisableTiming));
  HIPI(hipEventCreateWithFlags(&h->ev_join, hipEventDisableTiming));
  for (int st = 0; st < cfg->n_stages; st++) {
    HIPI(hipStreamCreateWithFlags(&h->sst[st], hipStreamNonBlocking));
    HIPI(hipEventCreateWithFlags(&h->ev_st[st], hipEventDisableTiming));
  }
  HIPI(hipHostMalloc((void**)&h->pinned, sizeof(spd_step_result) * (kLogCap + 1), hipHostMallocDefault));

  const spd_config& c = *cfg;
  Ctx& C = h->ctx;
  std::memset(&C, 0, sizeof(C));
  C.d = c.d_model;
  C.hq = c.n_q_heads;
  C.hkv = c.n_kv_heads;
  C.dh = c.head_dim;
  C.qdim = c.n_q_heads * c.head_dim;
  C.kvdim = c.n_kv_heads * c.head_dim;
  C.F = c.ffn_dim;
  C.V = c.vocab;
  C.L = c.n_layers;
  C.n = c.n_stages;
  C.ls = c.pdm_layers;
  C.page = c.page_size;
  C.chunk = lay.chunk;
  C.rows_wgs = default_rows_wgs(c);
  C.max_pages = lay.num_pages;
  C.max_splits = lay.max_splits;
  C.max_tokens = c.max_tokens;
  C.G = c.n_q_heads / c.n_kv_heads;
  C.eps = c.rms_eps;
  C.scale = (float)(1.0 / std::sqrt((double)c.head_dim));
  stage_bounds(c.n_layers, c.n_stages, C.beta);
  h->J = 0;
  for (int s = 0; s < c.n_stages; s++) h->J = std::max(h->J, C.beta[s + 1] - C.beta[s]);
  C.J = h->J;
  char* ws = h->ws;
  C.lay = (const LayerDesc*)(ws + lay.lay);
  C.embed = w->embed;
  C.lm_head = w->lm_head;
  C.pdm_V = cfg->pdm_vocab;
  C.pdm_head = cfg->pdm_vocab > 0 ? w->pdm_lm_head : w->lm_head;
  C.pdm_map = cfg->pdm_vocab > 0 ? w->pdm_vocab_map : nullptr;
  if (cfg->pdm_vocab > 0) {  // every draft id must name a target token (it is embedded when pushed)
    std::vector<int32_t> map(cfg->pdm_vocab);
    HIPI(hipMemcpy(map.data(), w->pdm_vocab_map, sizeof(int32_t) * map.size(), hipMemcpyDeviceToHost));
    for (int32_t t : map)
      if (t < 0 || t >= cfg->vocab) {
        h->err = "weights: pdm_vocab_map holds an id outside [0, vocab)";
        return fail(SPD_E_INVAL);
      }
  }
  C.w_in = w->pdm_in;
  C.final_norm = (const float*)w->final_norm;
  C.pdm_norm = (const float*)w->pdm_norm;
  C.page_table = (const int32_t*)(ws + lay.pt);
  C.rope = (const float2*)(ws + lay.rope);
  C.st = (DevState*)(ws + lay.state);
  C.tok = (int32_t*)(ws + lay.tok);
  C.forced = (int32_t*)(ws + lay.forced);
  C.log = (spd_step_result*)(ws + lay.log);
  C.resid = (float*)(ws + lay.resid);
  C.anchors = (float*)(ws + lay.anch);
  C.pdm_x = (float*)(ws + lay.pdmx);
  C.pf_x = (float*)(ws + lay.pfx);
  C.pf_anch = (float*)(ws + lay.pfanch);
  C.dbg_logits = (float*)(ws + lay.dbg);
  C.debug = 0;
  for (int s = 0; s < 2; s++) {
    BufSet& B = C.b[s];
    B.q = (float*)(ws + lay.q[s]);
    B.ao = (float*)(ws + lay.ao[s]);
    B.act = (float*)(ws + lay.act[s]);
    B.part = (float*)(ws + lay.part[s]);
    B.cnt = (int32_t*)(ws + lay.cnt[s]);
    B.rpart = (float*)(ws + lay.rpart[s]);
    B.rtick = (int32_t*)(ws + lay.rtick[s]);
    B.hkey = (unsigned long long*)(ws + lay.hkey[s]);
  }
  C.post_step = 0;
  C.sam.top_k = 0;
  C.sam.inv_temp = 1.0f;
  C.sam.u = (const float*)(ws + lay.su);
  C.sam.wlog = (float*)(ws + lay.swlog);
  C.sam.wlog_stride = lay.wlog_stride;
  C.sam.wgmax = (unsigned long long*)(ws + lay.swgmax);
  C.sam.q_ids = (int32_t*)(ws + lay.sqids);
  C.sam.q_p = (float*)(ws + lay.sqp);
  C.sam.q_cnt = (int32_t*)(ws + lay.sqcnt);
  C.sam.pq_ids = (int32_t*)(ws + lay.spq);
  C.sam.pq_p = (float*)(ws + lay.spq + sizeof(int32_t) * kMaxTopK);
  C.sam.pq_cnt = (int32_t*)(ws + lay.spq + (sizeof(int32_t) + sizeof(float)) * kMaxTopK);

  // layer table
  std::vector<LayerDesc> ld(c.n_layers + c.pdm_layers);
  for (int l = 0; l < c.n_layers + c.pdm_layers; l++) {
    const bool pdm = l >= c.n_layers;
    const spd_layer_weights& s = pdm ? w->pdm_layers[l - c.n_layers] : w->layers[l];
    LayerDesc& d = ld[l];
    d.wq = s.wq;
    d.wk = s.wk;
    d.wv = s.wv;
    d.wo = s.wo;
    d.wg = s.wg;
    d.wu = s.wu;
    d.wd = s.wd;
    d.attn_norm = (const float*)s.attn_norm;
    d.mlp_norm = (const float*)s.mlp_norm;
    d.kv = pdm ? (void*)(ws + lay.pkv + lay.kv_layer_bytes * (l - c.n_layers))
               : (void*)(ws + lay.kv + lay.kv_layer_bytes * l);
  }
  // RoPE table: angle pos * base^(-2j/dh) and its cos/sin in double precision, rounded to fp32
  const int half = c.head_dim / 2;
  std::vector<float> rope((size_t)c.max_tokens * half * 2);
  for (int j = 0; j < half; j++) {
    const double inv = std::pow((double)c.rope_base, -2.0 * j / c.head_dim);
    for (int p = 0; p < c.max_tokens; p++) {
      const double ang = (double)p * inv;
      rope[((size_t)p * half + j) * 2] = (float)std::cos(ang);
      rope[((size_t)p * half + j) * 2 + 1] = (float)std::sin(ang);
    }
  }
  // page table: logical page i -> physical page, in order or seeded-shuffled
  h->page_table.resize(lay.num_pages);
  for (int i = 0; i < lay.num_pages; i++) h->page_table[i] = i;
  if (c.page_seed) {
    std::mt19937_64 rng(c.page_seed);
    for (int i = lay.num_pages - 1; i > 0; i--) {
      const int j = (int)(rng() % (uint64_t)(i + 1));
      std::swap(h->page_table[i], h->page_table[j]);
    }
  }
  h->layer_desc = ld;
  HIPI(hipMemcpyAsync(ws + lay.lay, ld.data(), sizeof(LayerDesc) * ld.size(), hipMemcpyHostToDevice, h->main));
  HIPI(hipMemcpyAsync(ws + lay.rope, rope.data(), sizeof(float) * rope.size(), hipMemcpyHostToDevice, h->main));
  HIPI(hipMemcpyAsync(ws + lay.pt, h->page_table.data(), sizeof(int32_t) * lay.num_pages, hipMemcpyHostToDevice,
                      h->main));
  HIPI(hipMemsetAsync(ws + lay.state, 0, sizeof(DevState), h->main));
  HIPI(hipMemsetAsync(ws + lay.tok, 0, sizeof(int32_t) * (c.max_tokens + 8), h->main));
  HIPI(hipMemsetAsync(ws + lay.forced, 0xff, sizeof(int32_t) * (c.max_tokens + 8), h->main));
  for (int s = 0; s < 2; s++) HIPI(hipMemsetAsync(ws + lay.cnt[s], 0, sizeof(int32_t) * kMaxStages * c.n_kv_heads, h->main));
  for (int s = 0; s < 2; s++) HIPI(hipMemsetAsync(ws + lay.rtick[s], 0, sizeof(int32_t) * kRowSplitCols, h->main));
  for (int s = 0; s < 2; s++) HIPI(hipMemsetAsync(ws + lay.hkey[s], 0, sizeof(unsigned long long), h->main));
  HIPI(hipMemsetAsync(ws + lay.sqcnt, 0, sizeof(int32_t) * c.n_stages, h->main));
  HIPI(hipMemsetAsync(ws + lay.spq, 0, (sizeof(int32_t) + sizeof(float)) * kMaxTopK + sizeof(int32_t), h->main));
  HIPI(hipStreamSynchronize(h->main));
#undef HIPI
  *out = h;
  return SPD_OK;
}

static void drop_graph(spd_handle* h);
static spd_status run_one_step(spd_handle* h, int forced_override);

spd_status spd_set_step_kernel(spd_handle* h, int32_t mode, int32_t grid, int32_t groups) {
  if (!h || (mode != 0 && mode != 2) || grid < 0 || grid > 65535 || groups < -1 || groups > kMaxStages)
    return SPD_E_INVAL;
  h->step_mode = mode;
  h->ctx.stream_wgs = grid;  // 0: default
  if (mode == 2 && groups >= 0) h->stage_groups = groups;
  drop_graph(h);  // the captured launches change
  return SPD_OK;
}

static spd_status refuse(spd_handle* h, const char* why) {
  h->err = why;
  return SPD_E_INVAL;
}

spd_status spd_set_sampling(spd_handle* h, int32_t top_k, float temperature, const float* uniforms,
                            int32_t positions) {
  if (!h) return SPD_E_INVAL;
  if (h->hstate != H_INIT) return SPD_E_STATE;
  if (top_k == 0) {
    h->ctx.sam.top_k = 0;
    drop_graph(h);
    return SPD_OK;
  }
  if (top_k < 0 || top_k > kMaxTopK) return refuse(h, "top_k must be in [0, 64]");
  if (!(temperature > 0.f) || !std::isfinite(temperature)) return refuse(h, "temperature must be > 0");
  if (!uniforms || positions != h->cfg.max_tokens)
    return refuse(h, "uniforms must hold 3 * max_tokens values");
  for (size_t i = 0; i < (size_t)3 * positions; i++)
    if (!(uniforms[i] >= 0.f && uniforms[i] < 1.f)) return refuse(h, "uniforms must lie in [0, 1)");
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->main));
  HIPC(hipMemcpy(h->ws + h->lay.su, uniforms, sizeof(float) * 3 * (size_t)positions, hipMemcpyHostToDevice));
  h->ctx.sam.top_k = top_k;
  h->ctx.sam.inv_temp = 1.0f / temperature;
  drop_graph(h);  // the captured launches change
  return SPD_OK;
}

spd_status spd_set_pdm_schedule(spd_handle* h, int32_t post_step) {
  if (!h || (post_step != 0 && post_step != 1)) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->main));
  h->ctx.post_step = post_step;
  drop_graph(h);  // the captured launches change
  return SPD_OK;
}

spd_status spd_set_pdm_enabled(spd_handle* h, int32_t on) {
  if (!h) return SPD_E_INVAL;
  h->pdm_on = on ? 1 : 0;
  drop_graph(h);  // the captured launches change
  return SPD_OK;
}

spd_status spd_probe_hbm_read(const void* buf, size_t bytes, float* sink, int32_t reps, void* stream, double* ms) {
  if (!buf || !sink || !ms || bytes < 16 || reps < 1 || ((uintptr_t)buf & 15)) return SPD_E_INVAL;
  hipStream_t s = (hipStream_t)stream;
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) return SPD_E_HIP;
  launch_read_probe(buf, bytes / 16, sink, s);  // warm-up
  (void)hipEventRecord(e0, s);
  for (int i = 0; i < reps; i++) launch_read_probe(buf, bytes / 16, sink, s);
  (void)hipEventRecord(e1, s);
  hipError_t e = hipEventSynchronize(e1);
  float t = 0.f;
  if (e == hipSuccess) e = hipEventElapsedTime(&t, e0, e1);
  (void)hipEventDestroy(e0);
  (void)hipEventDestroy(e1);
  if (e != hipSuccess) return SPD_E_HIP;
  *ms = (double)t / reps;
  return SPD_OK;
}

spd_status spd_set_pdm_placement(spd_handle* h, int32_t place) {
  if (!h || place < 0 || place > 3) return SPD_E_INVAL;
  h->pdm_place = place;
  drop_graph(h);  // the captured launches change
  return SPD_OK;
}

spd_status spd_set_pdm_grid(spd_handle* h, int32_t wgs) {
  if (!h || wgs < 0 || wgs > 65535) return SPD_E_INVAL;
  h->ctx.rows_wgs = wgs > 0 ? wgs : default_rows_wgs(h->cfg);
  drop_graph(h);  // kernel arguments changed
  return SPD_OK;
}

spd_status spd_set_kernel_trace(spd_handle* h, int32_t on) {
  if (!h) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->pdm));
  HIPC(hipStreamSynchronize(h->main));
  h->ctx.ktrace = on ? (unsigned long long*)(h->ws + h->lay.ktrace) : nullptr;
  drop_graph(h);  // kernel arguments changed
  return SPD_OK;
}

spd_status spd_step_plan_info(spd_handle* h, int32_t* info) {
  if (!h || !info) return SPD_E_INVAL;
  for (int i = 0; i < 8; i++) info[i] = 0;
  info[0] = h->lay.J;
  int khz = 0;
  HIPC(hipDeviceGetAttribute(&khz, hipDeviceAttributeWallClockRate, h->dev));
  info[1] = khz;
  info[2] = h->lay.nkslots;
  info[3] = h->cfg.n_stages;
  info[4] = h->step_mode == 2 ? std::min(h->stage_groups > 0 ? h->stage_groups : kStageGroupsDefault,
                                         h->cfg.n_stages)
                              : 1;
  info[5] = h->pdm_place;
  return SPD_OK;
}

spd_status spd_set_debug(spd_handle* h, int32_t on) {
  if (!h) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->pdm));
  HIPC(hipStreamSynchronize(h->main));
  h->ctx.debug = on ? 1 : 0;
  drop_graph(h);  // kernel arguments changed
  return SPD_OK;
}

static spd_status fetch_state(spd_handle* h) {
  HIPC(hipMemcpyAsync(h->pinned, &h->ctx.st->res, sizeof(spd_step_result), hipMemcpyDeviceToHost, h->main));
  HIPC(hipStreamSynchronize(h->main));
  const spd_step_result& r = h->pinned[0];
  h->c = r.committed_len;
  h->a = r.inflight;
  h->bound = (long long)h->c + h->a;
  h->unsynced = 0;
  return SPD_OK;
}

static spd_status ensure_synced(spd_handle* h) {
  if (!h->unsynced) return SPD_OK;
  HIPC(hipStreamSynchronize(h->pdm));
  return fetch_state(h);
}

spd_status spd_prefill(spd_handle* h, const int32_t* prompt, int32_t len, int32_t* first_token) {
  if (!h || !prompt || len < 1) return SPD_E_INVAL;
  if (h->hstate != H_INIT) return SPD_E_STATE;
  if (len + h->cfg.n_stages + 1 > h->cfg.max_tokens) return SPD_E_CAPACITY;
  for (int i = 0; i < len; i++)
    if (prompt[i] < 0 || prompt[i] >= h->cfg.vocab) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipMemcpyAsync(h->ctx.tok, prompt, sizeof(int32_t) * len, hipMemcpyHostToDevice, h->main));
  spd_status st = h->bf16 ? enqueue_prefill<uint16_t>(h, len) : enqueue_prefill<float>(h, len);
  if (st != SPD_OK) return st;
  int32_t y = 0;
  HIPC(hipMemcpyAsync(&h->pinned[0].target_argmax, &h->ctx.st->y, sizeof(int32_t), hipMemcpyDeviceToHost, h->main));
  HIPC(hipStreamSynchronize(h->main));
  y = h->pinned[0].target_argmax;
  h->c = len;
  h->a = 1;
  h->bound = len + 1;
  h->prompt_len = len;
  h->hstate = H_READY;
  if (first_token) *first_token = y;
  return SPD_OK;
}

spd_status spd_step(spd_handle* h, const int32_t* forced_draft, spd_step_result* out) {
  if (!h) return SPD_E_INVAL;
  if (h->hstate != H_READY) return SPD_E_STATE;
  if (forced_draft && (*forced_draft < 0 || *forced_draft >= h->cfg.vocab)) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  spd_status sy = ensure_synced(h);
  if (sy != SPD_OK) return sy;
  if (h->c + h->a >= h->cfg.max_tokens) return SPD_E_CAPACITY;
  spd_status st = run_one_step(h, forced_draft ? *forced_draft : -1);
  if (st != SPD_OK) return st;
  st = fetch_state(h);
  if (st != SPD_OK) return st;
  const spd_step_result r = h->pinned[0];
  if (r.decision == SPD_REJECT && !h->cfg.auto_rollback) h->hstate = H_PENDING;
  if (out) *out = r;
  return SPD_OK;
}

static void drop_graph(spd_handle* h) {
  if (h->gexec) (void)hipGraphExecDestroy(h->gexec);
  if (h->gexec_multi) (void)hipGraphExecDestroy(h->gexec_multi);
  h->gexec = nullptr;
  h->gexec_multi = nullptr;
}

// Capture `steps` consecutive steps (each the launches of enqueue_step) into one executable graph.
// Nothing a step enqueues depends on host state, so the steps chain on the device alone.
static spd_status capture_steps(spd_handle* h, int steps, hipGraphExec_t* out) {
  hipGraph_t g = nullptr;
  HIPC(hipStreamBeginCapture(h->main, hipStreamCaptureModeRelaxed));
  spd_status st = SPD_OK;
  for (int i = 0; i < steps && st == SPD_OK; i++)
    st = h->bf16 ? enqueue_step<uint16_t>(h, -1) : enqueue_step<float>(h, -1);
  hipError_t e = hipStreamEndCapture(h->main, &g);
  if (st != SPD_OK) {
    if (g) (void)hipGraphDestroy(g);
    return st;
  }
  if (e != hipSuccess) {
    h->err = std::string("hipStreamEndCapture: ") + hipGetErrorString(e);
    return SPD_E_HIP;
  }
  e = hipGraphInstantiate(out, g, nullptr, nullptr, 0);
  (void)hipGraphDestroy(g);
  if (e != hipSuccess) {
    *out = nullptr;
    h->err = std::string("hipGraphInstantiate: ") + hipGetErrorString(e);
    return SPD_E_HIP;
  }
  return SPD_OK;
}

// One step: a replay of the captured step graph when graph mode is on (and no per-step override or
// kernel timing is active), else the launches themselves.
static spd_status run_one_step(spd_handle* h, int forced_override) {
  const bool graph = h->use_graph && forced_override < 0 && h->timed_kernel == 0;
  if (!graph) return h->bf16 ? enqueue_step<uint16_t>(h, forced_override) : enqueue_step<float>(h, forced_override);
  if (!h->gexec) {
    spd_status st = capture_steps(h, 1, &h->gexec);
    if (st != SPD_OK) return st;
  }
  HIPC(hipGraphLaunch(h->gexec, h->main));
  return SPD_OK;
}

spd_status spd_set_graph_steps(spd_handle* h, int32_t steps) {
  if (!h || steps < 1 || steps > 16) return SPD_E_INVAL;
  h->graph_steps = steps;
  drop_graph(h);
  return SPD_OK;
}

spd_status spd_set_graph(spd_handle* h, int32_t on) {
  if (!h) return SPD_E_INVAL;
  h->use_graph = on ? 1 : 0;
  if (!on) drop_graph(h);
  return SPD_OK;
}

spd_status spd_run_steps(spd_handle* h, int32_t count, spd_step_result* log) {
  if (!h || count < 0) return SPD_E_INVAL;
  if (h->hstate != H_READY || !h->cfg.auto_rollback) return SPD_E_STATE;
  if (count > kLogCap && log) return SPD_E_INVAL;
  if (h->bound + count > h->cfg.max_tokens) return SPD_E_CAPACITY;
  HIPC(hipSetDevice(h->dev));
  int i = 0;
  if (h->use_graph && h->timed_kernel == 0 && h->graph_steps > 1) {  // whole multi-step graphs first
    for (; i + h->graph_steps <= count; i += h->graph_steps) {
      if (!h->gexec_multi) {
        spd_status st = capture_steps(h, h->graph_steps, &h->gexec_multi);
        if (st != SPD_OK) return st;
      }
      HIPC(hipGraphLaunch(h->gexec_multi, h->main));
    }
  }
  for (; i < count; i++) {
    spd_status st = run_one_step(h, -1);
    if (st != SPD_OK) return st;
  }
  h->bound += count;
  h->unsynced = 1;
  if (log) {
    spd_status st = fetch_state(h);
    if (st != SPD_OK) return st;
    const int last = h->pinned[0].step_index;
    // the ring entries of the last `count` steps: one contiguous run, or two where it wraps
    const int start = (last - count) % kLogCap;
    const int n1 = std::min(count, kLogCap - start);
    if (n1 > 0)
      HIPC(hipMemcpyAsync(&h->pinned[1], h->ctx.log + start, sizeof(spd_step_result) * n1, hipMemcpyDeviceToHost,
                          h->main));
    if (count > n1)
      HIPC(hipMemcpyAsync(&h->pinned[1 + n1], h->ctx.log, sizeof(spd_step_result) * (count - n1),
                          hipMemcpyDeviceToHost, h->main));
    HIPC(hipStreamSynchronize(h->main));
    for (int i = 0; i < count; i++) log[i] = h->pinned[1 + i];
  }
  return SPD_OK;
}

spd_status spd_sync(spd_handle* h, spd_step_result* last) {
  if (!h) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->pdm));
  if (h->hstate == H_INIT) {
    HIPC(hipStreamSynchronize(h->main));
    return SPD_OK;
  }
  spd_status st = fetch_state(h);
  if (st != SPD_OK) return st;
  if (last) *last = h->pinned[0];
  return SPD_OK;
}

spd_status spd_rollback(spd_handle* h, int32_t keep_len, int32_t reseed_token) {
  if (!h) return SPD_E_INVAL;
  if (h->hstate == H_INIT) return SPD_E_STATE;
  if (reseed_token < 0 || reseed_token >= h->cfg.vocab) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  spd_status sy = ensure_synced(h);
  if (sy != SPD_OK) return sy;
  if (keep_len < h->prompt_len || keep_len > h->c) return SPD_E_INVAL;
  if (keep_len + 1 >= h->cfg.max_tokens) return SPD_E_CAPACITY;
  HIPC(hipStreamSynchronize(h->pdm));
  launch_reseed(h->ctx, keep_len, reseed_token, -1, h->main, h->bf16);
  spd_status st = launch_check(h, "rollback");
  if (st != SPD_OK) return st;
  HIPC(hipStreamSynchronize(h->main));
  h->c = keep_len;
  h->a = 1;
  h->bound = keep_len + 1;
  h->hstate = H_READY;
  return SPD_OK;
}

spd_status spd_set_forced_drafts(spd_handle* h, const int32_t* table, int32_t first_pos, int32_t len) {
  if (!h || (!table && len > 0) || first_pos < 0 || len < 0) return SPD_E_INVAL;
  if ((long long)first_pos + len > h->cfg.max_tokens) return SPD_E_CAPACITY;
  for (int i = 0; i < len; i++)
    if (table[i] >= h->cfg.vocab) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->main));
  if (len) HIPC(hipMemcpy(h->ctx.forced + first_pos, table, sizeof(int32_t) * len, hipMemcpyHostToDevice));
  return SPD_OK;
}

spd_status spd_clear_forced_drafts(spd_handle* h) {
  if (!h) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->main));
  HIPC(hipMemset(h->ctx.forced, 0xff, sizeof(int32_t) * (h->cfg.max_tokens + 8)));
  return SPD_OK;
}

spd_status spd_read_debug(spd_handle* h, int32_t what, void* host, size_t bytes) {
  if (!h || !host) return SPD_E_INVAL;
  const spd_config& c = h->cfg;
  const void* src = nullptr;
  size_t need = 0;
  switch (what) {
    case SPD_DBG_RESID: src = h->ctx.resid; need = sizeof(float) * c.n_stages * c.d_model; break;
    case SPD_DBG_ANCHORS: src = h->ctx.anchors; need = sizeof(float) * c.n_stages * c.n_stages * c.d_model; break;
    case SPD_DBG_PDM_HIDDEN: src = h->ctx.pdm_x; need = sizeof(float) * kMaxRows * c.d_model; break;
    case SPD_DBG_EXIT_LOGITS: src = h->ctx.dbg_logits; need = sizeof(float) * c.vocab; break;
    case SPD_DBG_PDM_LOGITS:
      src = h->ctx.dbg_logits + c.vocab;
      need = sizeof(float) * (c.pdm_vocab > 0 ? c.pdm_vocab : c.vocab);
      break;
    case SPD_DBG_TOKENS: src = h->ctx.tok; need = sizeof(int32_t) * c.max_tokens; break;
    case SPD_DBG_STATE: src = nullptr; need = sizeof(int32_t) * 4; break;
    case SPD_DBG_QDIST: src = nullptr; need = sizeof(int32_t) * c.n_stages * (1 + 2 * kMaxTopK); break;
    case SPD_DBG_KTRACE:
      src = h->ws + h->lay.ktrace;
      need = sizeof(unsigned long long) * 2 * (size_t)h->lay.nkslots;
      break;
    default: return SPD_E_INVAL;
  }
  if (bytes != need) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->pdm));
  HIPC(hipStreamSynchronize(h->main));
  if (what == SPD_DBG_STATE) {
    DevState s;
    HIPC(hipMemcpy(&s, h->ctx.st, sizeof(DevState), hipMemcpyDeviceToHost));
    int32_t* o = (int32_t*)host;
    o[0] = s.c;
    o[1] = s.a;
    o[2] = s.prompt_len;
    o[3] = s.nsteps;
    return SPD_OK;
  }
  if (what == SPD_DBG_QDIST) {
    const int n = c.n_stages;
    char* o = (char*)host;
    HIPC(hipMemcpy(o, h->ctx.sam.q_cnt, sizeof(int32_t) * n, hipMemcpyDeviceToHost));
    HIPC(hipMemcpy(o + sizeof(int32_t) * n, h->ctx.sam.q_ids, sizeof(int32_t) * n * kMaxTopK, hipMemcpyDeviceToHost));
    HIPC(hipMemcpy(o + sizeof(int32_t) * n * (1 + kMaxTopK), h->ctx.sam.q_p, sizeof(float) * n * kMaxTopK,
                   hipMemcpyDeviceToHost));
    return SPD_OK;
  }
  HIPC(hipMemcpy(host, src, need, hipMemcpyDeviceToHost));
  return SPD_OK;
}

spd_status spd_read_kv(spd_handle* h, int32_t pdm, int32_t layer, int32_t pos0, int32_t count, void* host_k,
                       void* host_v) {
  if (!h || !host_k || !host_v || count < 0 || pos0 < 0) return SPD_E_INVAL;
  const spd_config& c = h->cfg;
  if (layer < 0 || layer >= (pdm ? c.pdm_layers : c.n_layers)) return SPD_E_INVAL;
  if ((long long)pos0 + count > c.max_tokens) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->pdm));
  HIPC(hipStreamSynchronize(h->main));
  const size_t esz = h->bf16 ? 2 : 4;
  const int P = c.page_size, hkv = c.n_kv_heads, dh = c.head_dim;
  const size_t page_bytes = (size_t)2 * hkv * P * dh * esz;
  const char* base = h->ws + (pdm ? h->lay.pkv : h->lay.kv) + h->lay.kv_layer_bytes * layer;
  std::vector<char> pg(page_bytes);
  int cur = -1;
  for (int p = pos0; p < pos0 + count; p++) {
    const int lp = p / P;
    if (lp != cur) {
      HIPC(hipMemcpy(pg.data(), base + (size_t)h->page_table[lp] * page_bytes, page_bytes, hipMemcpyDeviceToHost));
      cur = lp;
    }
    for (int g = 0; g < hkv; g++) {
      const size_t ko = ((size_t)g * P + (p % P)) * dh * esz;
      const size_t vo = ko + (size_t)hkv * P * dh * esz;
      const size_t oo = ((size_t)(p - pos0) * hkv + g) * dh * esz;
      std::memcpy((char*)host_k + oo, pg.data() + ko, dh * esz);
      std::memcpy((char*)host_v + oo, pg.data() + vo, dh * esz);
    }
  }
  return SPD_OK;
}

spd_status spd_set_kernel_timing(spd_handle* h, int32_t kernel, int32_t first_slot) {
  if (!h || kernel < 0 || kernel > SPD_K_SPANS || first_slot < 0) return SPD_E_INVAL;
  h->timed_kernel = kernel;
  h->timed_first_slot = first_slot;
  return SPD_OK;
}

spd_status spd_kernel_timing(spd_handle* h, double* total_ms, int32_t* launches) {
  if (!h || !total_ms || !launches) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->main));
  double tot = 0.0;
  for (size_t i = 0; i + 1 < h->tev_used; i += 2) {
    float ms = 0.f;
    HIPC(hipEventElapsedTime(&ms, h->tev[i], h->tev[i + 1]));
    tot += ms;
  }
  *total_ms = tot;
  *launches = (int32_t)(h->tev_used / 2);
  h->tev_used = 0;
  return SPD_OK;
}

spd_status spd_span_timing(spd_handle* h, double* stage_ms, double* pdm_ms, double* late_ms, int32_t* steps) {
  if (!h || !stage_ms || !pdm_ms || !late_ms || !steps) return SPD_E_INVAL;
  HIPC(hipSetDevice(h->dev));
  HIPC(hipStreamSynchronize(h->pdm));
  HIPC(hipStreamSynchronize(h->main));
  double st = 0.0, pd = 0.0, late = 0.0;
  for (size_t i = 0; i + 3 <= h->sev_used; i += 3) {
    float a = 0.f, b = 0.f;
    HIPC(hipEventElapsedTime(&a, h->sev[i], h->sev[i + 2]));
    HIPC(hipEventElapsedTime(&b, h->sev[i], h->sev[i + 1]));
    st += a;
    pd += b;
    late += b > a ? (double)(b - a) : 0.0;
  }
  *stage_ms = st;
  *pdm_ms = pd;
  *late_ms = late;
  *steps = (int32_t)(h->sev_used / 3);
  h->sev_used = 0;
  return SPD_OK;
}

void spd_destroy(spd_handle* h) {
  if (!h) return;
  drop_graph(h);
  for (hipEvent_t e : h->tev) (void)hipEventDestroy(e);
  for (hipEvent_t e : h->sev) (void)hipEventDestroy(e);
  if (h->main) (void)hipStreamSynchronize(h->main);
  if (h->pdm) (void)hipStreamSynchronize(h->pdm);
  for (int st = 0; st < kMaxStages; st++) {
    if (h->sst[st]) (void)hipStreamSynchronize(h->sst[st]);
    if (h->ev_st[st]) (void)hipEventDestroy(h->ev_st[st]);
    if (h->sst[st]) (void)hipStreamDestroy(h->sst[st]);
  }
  if (h->ev_fork) (void)hipEventDestroy(h->ev_fork);
  if (h->ev_join) (void)hipEventDestroy(h->ev_join);
  if (h->pinned) (void)hipHostFree(h->pinned);
  delete h;
}

}  // extern "C"
