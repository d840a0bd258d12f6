// Internal layout shared by the host runtime and the gfx950 kernels. Not part of the C ABI.
#pragma once
#include <stddef.h>
#include <stdint.h>

#include "spd.h"

namespace spd {

constexpr int kMaxStages = 8;   // n
constexpr int kMaxRows = 8;     // rows of one row-block launch (PDM rows, prefill chunk)
// Uncapped row-block GEMVs (prefill chunks) whose rows' input vectors take more LDS than kRowLdsBudget
// at full width run K-split: chunks of kRowSplitK inputs, at most kRowSplitCols workgroup columns.
constexpr int kRowSplitK = 1024;
constexpr int kRowLdsBudget = 64 * 1024;
constexpr int kRowSplitCols = 1024;
constexpr int kMaxPdmLayers = 4;
constexpr int kWG = 256;        // threads per workgroup in every kernel
constexpr int kLogCap = 4096;   // step log ring
constexpr int kMaxSplits = 64;  // attention key splits per (row, KV head)

// One decoder layer as the kernels see it. KV pool of the layer: [pages][2][Hkv][page][dh].
struct LayerDesc {
  const void* wq;
  const void* wk;
  const void* wv;
  const void* wo;
  const void* wg;
  const void* wu;
  const void* wd;
  const float* attn_norm;
  const float* mlp_norm;
  void* kv;
};

// Device-resident decoding state; every kernel of a step reads the pre-step c and a from here and
// only the verify kernel (last in the step) changes them.
struct DevState {
  int32_t c;           // positions that have passed all layers
  int32_t a;           // in-flight tokens, positions c..c+a-1 (0 while a rollback is pending)
  int32_t prompt_len;
  int32_t pending;     // 1: a REJECT waits for spd_rollback
  int32_t nsteps;
  int32_t y;           // target argmax of this step's exiting token
  int32_t pdm_draft;   // PDM argmax of this step
  spd_step_result res; // last step
  int32_t head_ticket; // workgroups of the fused LM head + verify launch that are done (zero at rest)
  int32_t pad1[5];
};

// Scratch of one compute stream. The target path and the PDM each own one, so the two streams
// never share scratch.
struct BufSet {
  float* q;         // [8][Hq*dh] rotated queries (row index = group for stage launches)
  float* ao;        // [8][Hq*dh] attention outputs
  float* act;       // [8][F] SwiGLU activations
  float* part;      // attention split partials
  int32_t* cnt;     // per (stage, KV head) split tickets of the decode attention; zero at rest
  float* rpart;     // K-split row GEMV records (chunk dot products, sums of squares)
  int32_t* rtick;   // K-split row GEMV tickets, one per workgroup column; zero at rest
  // LM-head argmax of this stream's row: the maximum over the vocabulary of a 64-bit key that
  // orders (logit descending, index ascending); zero at rest (reset by its reader)
  unsigned long long* hkey;
};

// Sublayers of a layer slot, in launch order (the launch trace's slot index uses the same order).
enum StepKind { SK_QKV = 0, SK_ATTN = 1, SK_OPROJ = 2, SK_GATEUP = 3, SK_DOWN = 4 };
// Stage groups: the stages of a step are spread over this many streams (groups of consecutive
// stages). With the PDM's stream, more than four parallel chains per step make the runtime run one
// chain after another; two groups keep every chain running from the fork.
constexpr int kStageGroupsDefault = 2;
constexpr int kStreamWGs = 1024;  // workgroups of one streaming stage launch (all its stages)
// PDM row-block GEMV launches run beside the stage compute: a few workgroups, so that most CUs (and
// their LDS) stay with the stage launches.
constexpr int kRowsWGsDefault = 32;
// Sampled decoding (top-k, temperature): at most this many tokens per distribution; a sampled
// LM-head launch has at most kSampleWGs workgroups (each leaves one maximum per row), and its
// selection keeps up to kSelCap candidates in LDS (more go through a slower pass over memory).
constexpr int kMaxTopK = 64;
constexpr int kSampleWGs = 1024;
constexpr int kSelCap = 1024;
// Sampled decoding state. The sampled LM-head launch leaves every logit of its rows in wlog, one
// region of cmax = 2*ceil(pairs / waves) floats per wave (entry i of wave w is vocabulary row
// 2*(w + (i/2)*waves) + i%2), and each workgroup's best key per row in wgmax; q_* hold the draft
// distribution of every in-flight token (row = position mod n) until its acceptance test.
struct Sampler {
  int top_k;                  // 0: greedy decoding
  float inv_temp;             // 1 / temperature
  const float* u;             // [max_tokens][3]: u_draft, u_accept, u_resample of each position
  float* wlog;                // [2][wlog_stride]: row 0 the exit (or prefill) row, row 1 the PDM row
  int wlog_stride;            // floats per row, >= V + 8 * kSampleWGs
  unsigned long long* wgmax;  // [2][kSampleWGs]
  int32_t* q_ids;             // [n][kMaxTopK]
  float* q_p;                 // [n][kMaxTopK]
  int32_t* q_cnt;             // [n]
  // the draft module's top-k distribution when its row has its own head pass (target ids)
  int32_t* pq_ids;            // [kMaxTopK]
  float* pq_p;                // [kMaxTopK]
  int32_t* pq_cnt;            // [1]
};

struct Ctx {
  // shapes
  int d, hq, hkv, dh, qdim, kvdim, F, V, L, n, ls, page, chunk, max_pages, max_splits, max_tokens;
  int G;            // query heads per KV head
  float eps, scale; // RMSNorm eps, 1/sqrt(dh)
  int beta[kMaxStages + 1];
  // weights and tables
  const LayerDesc* lay;   // [L + ls]: target layers then PDM layers
  const void* embed;
  const void* lm_head;
  const void* w_in;
  const float* final_norm;
  const float* pdm_norm;
  const void* pdm_head;      // the PDM's own LM head [pdm_V x d], or the shared lm_head (pdm_V == 0)
  const int32_t* pdm_map;    // pdm_V > 0: target token of each draft id
  int pdm_V;                 // 0: shared head
  const int32_t* page_table;
  const float2* rope;     // [max_tokens][dh/2] (cos, sin)
  // state
  DevState* st;
  int32_t* tok;           // [max_tokens + 8]
  int32_t* forced;        // [max_tokens + 8], -1 = no override
  spd_step_result* log;   // [kLogCap]
  // activations
  float* resid;     // [n][d] in-flight residual streams, row q mod n
  float* anchors;   // [n][n][d] row q mod n, anchor j
  float* pdm_x;     // [8][d] PDM residual rows
  float* pf_x;      // [8][d] prefill chunk residual rows
  float* pf_anch;   // [8][n][d] prefill chunk anchors
  float* dbg_logits;// [2][V]
  int debug;
  BufSet b[2];      // 0: target stream, 1: PDM stream
  unsigned long long* ktrace;  // null, or the launch trace: per slot (first start, last end) wall clock
  int stream_wgs;   // workgroups of one streaming stage launch (all its stages)
  int rows_wgs;     // at most this many workgroups per row-block (PDM) GEMV launch (0: no cap)
  int J;            // layer slots per step (longest stage)
  Sampler sam;      // sampled decoding (sam.top_k == 0: greedy)
  int post_step;    // 1: the PDM reads the features after the step's stage compute (one stage deeper)
};

// Which rows a launch works on.
//   kind 0 (stage launch): group g = stage s = stage0 + g, one row: the token at depth s, position c+a-1-s,
//            layer beta_s + slot (inactive if s >= a or the stage has fewer layers).
//   kind 1 (row block): one group of `nrows` rows at positions pos0+i through layer `layer`;
//            nrows < 0 means "a" and pos0 < 0 means "c" read from the device state (PDM step).
struct Rows {
  int kind;
  int slot;
  int stage0;   // kind 0: group g of the launch is stage stage0 + g
  int nst;      // kind 0: stages in the launch (grid y, or z for attention)
  int layer;    // kind 1: index into Ctx::lay
  int nrows;
  int pos0;
  float* x;     // kind 1: residual rows [nrows][d]
  float* anch;  // kind 1: anchor capture base [rows][n][d] (null: none)
  int cap;      // kind 1: anchor index to capture after this layer (-1: none)
  int set;      // scratch set
  // kind 0: layer beta_s + slot of every stage s, passed with the launch so that weight loads need
  // no table lookup (all pointers null for a stage with no layer in this slot)
  LayerDesc ld[kMaxStages];
};

// Launchers (spd_kernels.hip). All are asynchronous on `stream`.
template <typename WT>
struct Launch {
  static void qkv(const Ctx& c, const Rows& r, void* stream);
  static void attn(const Ctx& c, const Rows& r, void* stream);
  static void oproj(const Ctx& c, const Rows& r, void* stream);
  static void gateup(const Ctx& c, const Rows& r, void* stream);
  static void down(const Ctx& c, const Rows& r, void* stream);
  // One decoder layer of a row block whose rows share the layer (the PDM's rows in a step, or a
  // prefill chunk; at most max_rows rows): streaming GEMVs applying each weight pair to all rows
  // (the down projection also captures the rows' anchor when r.anch and r.cap name one), and the
  // rows' decode attention. Five launches; the GEMV launches take at most cap_wgs workgroups (0: as
  // many as fit at once).
  static void rows_layer(const Ctx& c, const Rows& r, int max_rows, int cap_wgs, void* stream);
  // sublayer k (0 QKV, 1 attention, 2 O-proj, 3 gate/up, 4 down) of rows_layer
  static void rows_sublayer(const Ctx& c, const Rows& r, int max_rows, int k, int cap_wgs, void* stream);
  // PDM feature projection; prefill = 1: nrows rows of pf_anch at full depth.
  static void pdm_fc(const Ctx& c, int prefill, int nrows, void* stream);
  // LM head + argmax partials. src: 0 = target exit row (skipped unless a == n), 1 = PDM last row,
  // 2 = prefill row `row` of pf_x, 3 = exit row and PDM row in one pass. The kernel that follows
  // (verify / reseed) reduces the partials.
  static void head(const Ctx& c, int src, int row, void* stream);
  // The two-row head (src 3) and the verify of the step in one launch: the workgroup that finishes
  // the head last runs the verify.
  // two_rows 0: the exit row alone (src 0), the PDM's draft already left by its own head pass.
  static void head_verify(const Ctx& c, int two_rows, int forced_override, int auto_rb, void* stream);
  // Sampled decoding (c.sam.top_k > 0). src 3: the two-row head, then the top-k distributions, the
  // draft's draw and the rejection-sampling verify of the step, in one launch; src 2: prefill row
  // `row` and the draw of the token at position pos (published as the row's argmax key, which the
  // reseed that follows reads).
  static void head_sample(const Ctx& c, int src, int row, int pos, int forced_override, int auto_rb,
                          void* stream);
  static void embed_rows(const Ctx& c, int t0, int nrows, void* stream);
};
void launch_ktrace_reset(const Ctx& c, int nslots, void* stream);
// Streaming read of n16 16-byte blocks (a bandwidth probe); sink gets one float per workgroup.
void launch_read_probe(const void* buf, size_t n16, float* sink, void* stream);
constexpr int kReadProbeWGs = 2048;
// Events (hipEvent_t) that the next launches of this host thread record at their own start and end;
// nullptr turns it off.
void set_launch_events(void* start, void* stop);
void launch_reseed(const Ctx& c, int keep, int tok, int prompt_len, void* stream, int bf16);

}  // namespace spd
