/*
 * spd.h — C ABI of the single-GPU Speculative Pipeline Decoding (SPD) step for MI355X (gfx950).
 *
 * The calls follow the method's statement of decoding: a prompt is processed (prefill), then each
 * pipeline step advances every in-flight token of one sequence through one stage of the target
 * (Section 3.1, token-level pipeline), while the Pipeline Draft Module drafts the next token from
 * pre-step multi-depth features (Sections 3.2-3.3, Eq. input-seq, Eq. agg-main); when the pipeline
 * is full the oldest token exits and its logits verify the next in-flight token, with rollback on
 * a mismatch (Section 3.4).
 *
 * Conventions shared by every entry point:
 *   - Ownership: the caller owns all device memory (weights, workspace) and both streams; they must
 *     outlive the handle. The library never frees caller memory and allocates only small host
 *     buffers (pinned result staging) and two events per handle.
 *   - Pointers marked "device" are HIP device addresses on the current device; "host" pointers are
 *     ordinary host memory. hipStream_t arguments are passed as void*.
 *   - Errors: every call returns spd_status; no C++ exception crosses the ABI. SPD_E_INVAL: bad
 *     argument; SPD_E_STATE: call not legal in the handle's state; SPD_E_CAPACITY: max_tokens or the
 *     workspace is too small; SPD_E_HIP: a HIP call failed (spd_last_error() has the message). On
 *     SPD_E_INVAL, SPD_E_STATE and SPD_E_CAPACITY the handle is unchanged.
 *   - Threads: one handle is used by one host thread at a time.
 */
#ifndef SPD_H
#define SPD_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum spd_status {
  SPD_OK = 0,
  SPD_E_INVAL = 1,
  SPD_E_STATE = 2,
  SPD_E_CAPACITY = 3,
  SPD_E_HIP = 4
} spd_status;

/* Storage type of weights (norm gains are always fp32) and of the KV caches. */
typedef enum spd_dtype { SPD_F32 = 0, SPD_BF16 = 1 } spd_dtype;

/* Outcome of one step (Section 3.4): NONE while the pipeline is filling (no token exits),
 * ACCEPT when the exiting token's greedy successor equals the in-flight token behind it,
 * REJECT otherwise (caches roll back to the committed prefix and the target's token is reseeded). */
typedef enum spd_decision { SPD_NONE = 0, SPD_ACCEPT = 1, SPD_REJECT = 2 } spd_decision;

/* Model and run configuration. The target is a pre-norm dense decoder with grouped-query attention,
 * rotate-half RoPE, RMSNorm and a SwiGLU MLP, no biases, untied embedding and LM head. Limits:
 * d_model, n_q_heads*head_dim and ffn_dim are multiples of 8; head_dim is 64 or 128;
 * n_q_heads = G * n_kv_heads with G in {1, 2, 4, 8}; 1 <= n_stages <= min(8, n_layers);
 * 1 <= pdm_layers <= 4; page_size is 16. */
typedef struct spd_config {
  int32_t n_layers;      /* L */
  int32_t d_model;       /* d */
  int32_t n_q_heads;     /* Hq */
  int32_t n_kv_heads;    /* Hkv */
  int32_t head_dim;      /* dh */
  int32_t ffn_dim;       /* F */
  int32_t vocab;         /* V */
  float rms_eps;         /* RMSNorm epsilon */
  float rope_base;       /* RoPE base: theta_j = base^(-2j/dh) */
  int32_t dtype;         /* spd_dtype */
  int32_t n_stages;      /* SPD width n: stage s holds layers [floor(sL/n), floor((s+1)L/n)) */
  int32_t pdm_layers;    /* L_s, decoder layers of the PDM */
  int32_t page_size;     /* KV page, in tokens */
  int32_t max_tokens;    /* capacity in positions: prompt + generated + n */
  int32_t auto_rollback; /* 1: spd_step applies the rollback of a REJECT itself (needed for
                            spd_run_steps); 0: a REJECT leaves the handle waiting for spd_rollback */
  int32_t attn_chunk;    /* keys per attention split, a multiple of page_size; 0 picks it from
                            max_tokens. Results depend on it, so compare runs with equal values. */
  uint64_t page_seed;    /* 0: physical KV pages are handed out in order; else in an order
                            shuffled with this seed (exercises the page table) */
  int32_t fused_head;    /* 1: the draft module's LM head shares the exit token's pass over the
                            vocabulary (one two-row pass on main_stream after the draft module's
                            layers join); 0: the draft module runs its own pass on pdm_stream.
                            Both give the same draft. */
  int32_t pdm_vocab;     /* 0: the draft module shares the target's lm_head. > 0: it has its own LM
                            head over this many tokens (Section 4.1: smaller vocabulary), in
                            spd_weights.pdm_lm_head / pdm_vocab_map; at most vocab; needs
                            fused_head = 0 (the two heads stream different weights) */
} spd_config;

/* One decoder layer's weights, all device pointers, row-major [out x in]:
 * attn_norm, mlp_norm: fp32 [d]; wq: [Hq*dh x d]; wk, wv: [Hkv*dh x d]; wo: [d x Hq*dh];
 * wg, wu: [F x d]; wd: [d x F]. Matrices are in the config's dtype, 16-byte aligned. */
typedef struct spd_layer_weights {
  const void* attn_norm;
  const void* wq;
  const void* wk;
  const void* wv;
  const void* wo;
  const void* mlp_norm;
  const void* wg;
  const void* wu;
  const void* wd;
} spd_layer_weights;

/* All weights. `layers` and `pdm_layers` are HOST arrays (n_layers and pdm_layers entries) of device
 * pointers; they are copied during spd_init. embed, lm_head: [V x d]; final_norm, pdm_norm: fp32 [d];
 * pdm_in: [d x n*d], the PDM's feature projection (Eq. agg-main): column block j multiplies the
 * anchor H^{beta_j} (the input of stage j). With spd_config.pdm_vocab = 0 the PDM shares the target's
 * lm_head and the last two pointers are ignored; otherwise pdm_lm_head is [pdm_vocab x d] (the
 * config's dtype) and pdm_vocab_map device int32 [pdm_vocab]: draft id i stands for target token
 * pdm_vocab_map[i], each in [0, vocab) (checked at spd_init; SPD_E_INVAL otherwise). The PDM's
 * draft is pdm_vocab_map[argmax] (lowest draft id on ties). */
typedef struct spd_weights {
  const void* embed;
  const spd_layer_weights* layers;
  const void* final_norm;
  const void* lm_head;
  const void* pdm_in;
  const spd_layer_weights* pdm_layers;
  const void* pdm_norm;
  const void* pdm_lm_head;
  const int32_t* pdm_vocab_map;
} spd_weights;

/* Result of one step. Positions are 0-based. committed_len = c, the number of positions that have
 * passed all L layers; inflight = a, tokens in the pipeline at positions c..c+a-1. */
typedef struct spd_step_result {
  int32_t decision;       /* spd_decision */
  int32_t target_argmax;  /* y: greedy successor of the exiting token, -1 if none exited */
  int32_t draft;          /* token pushed at depth 0 (the PDM's draft unless forced); -1 on REJECT */
  int32_t pdm_draft;      /* the PDM's own argmax */
  int32_t exited_pos;     /* position that left the last stage, -1 if none */
  int32_t exited_token;   /* token at exited_pos (committed in an earlier step), -1 if none */
  int32_t verified_pos;   /* position judged this step, -1 if none */
  int32_t verified_token; /* token now committed at verified_pos (equals target_argmax) */
  int32_t committed_len;  /* c after the step */
  int32_t inflight;       /* a after the step (0 while a rollback is pending) */
  int32_t step_index;     /* steps taken since prefill, counting this one */
} spd_step_result;

typedef struct spd_handle spd_handle;

/* Bytes of device workspace spd_init needs for cfg (KV pools, page table, RoPE table, in-flight
 * activations and scratch). Host-only: touches no GPU. */
spd_status spd_workspace_size(const spd_config* cfg, size_t* bytes);

/* Stage boundaries beta_0..beta_n (host array of n_stages+1 ints), beta_s = floor(s*L/n)
 * (Section 3.1 uniform split, Section 4.1). Host-only. */
spd_status spd_stage_bounds(const spd_config* cfg, int32_t* beta);

/* Bind weights and workspace, build the tables (RoPE cos/sin in double precision rounded to fp32,
 * page table, layer table) and return a handle. workspace: device, >= spd_workspace_size bytes,
 * 256-byte aligned. main_stream runs the stage compute, pdm_stream the draft module (they must
 * differ; both default priority). */
spd_status spd_init(const spd_config* cfg, const spd_weights* w, void* workspace, size_t ws_bytes,
                    void* main_stream, void* pdm_stream, spd_handle** out);

/* Process the prompt (host int32[len], ids in [0, V)) through the target, keeping the stage-input
 * hidden states as PDM anchors, build the PDM KV over the prompt with full-depth features, and
 * place the target's greedy token x_len in flight at depth 0. Writes x_len to *first_token.
 * Legal once, right after spd_init. Synchronous. */
spd_status spd_prefill(spd_handle* h, const int32_t* prompt, int32_t len, int32_t* first_token);

/* One pipeline step (Section 3.1-3.4): PDM on pdm_stream over pre-step features, every active
 * stage on main_stream, exit + greedy verify when the pipeline is full. forced_draft (host, may be
 * NULL) replaces the PDM's draft for this step; the PDM still runs. Synchronous: returns after the
 * result is on the host. SPD_E_STATE before prefill or while a rollback is pending. */
spd_status spd_step(spd_handle* h, const int32_t* forced_draft, spd_step_result* out);

/* Keep positions < keep_len in every target and PDM cache, drop all in-flight work and put
 * reseed_token in flight at position keep_len, depth 0 (Section 3.4 with keep_len = t-n+1).
 * Requires prompt_len <= keep_len <= c and 0 <= reseed_token < V. */
spd_status spd_rollback(spd_handle* h, int32_t keep_len, int32_t reseed_token);

/* Per-position draft override table used by spd_step and spd_run_steps: for each position
 * first_pos+i with table[i] >= 0 the draft pushed at that position is table[i]. table: host. */
spd_status spd_set_forced_drafts(spd_handle* h, const int32_t* table, int32_t first_pos, int32_t len);
spd_status spd_clear_forced_drafts(spd_handle* h);

/* Sampled decoding (Section 3.4 under sampling; Section 4.1 samples at temperature 1 with top-k 50
 * and top-p 1.0). Every distribution is the softmax at `temperature` of the top_k largest logits
 * (lower index first among equal logits). The PDM's draft is drawn from its distribution q; when the
 * exiting token's distribution p judges the in-flight successor x, x is kept iff
 * u_accept * q(x) < p(x) (probability min(1, p(x)/q(x))), else the committed token is drawn from
 * max(0, p - q) normalised (from p if that has no mass) and reseeded, so the output follows p. A forced
 * draft has q = delta. The prompt's first token is drawn from p. Draws take the inverse CDF in
 * value-descending order: the first i with u * sum < cumsum_i.
 * uniforms: host float[3 * positions], positions == max_tokens; entry 3*pos + j is position pos's
 * u_draft (j = 0), u_accept (1) and u_resample (2), each in [0, 1); copied during the call.
 * top_k in [1, 64] turns sampling on, with either head form: the two-row pass selects both
 * distributions in its last workgroup; otherwise the draft module's own pass (shared or own head)
 * selects q and leaves it for the exit row's pass, which selects p and verifies. top_k = 0 returns
 * to greedy decoding (uniforms may then be NULL). Legal only before spd_prefill (SPD_E_STATE
 * afterwards); SPD_E_INVAL for other top_k, a temperature that is not finite and > 0, a uniforms
 * array of another length or a value outside [0, 1). In a sampled step
 * spd_step_result.target_argmax and verified_token hold the committed token and pdm_draft the
 * PDM's own draw. */
spd_status spd_set_sampling(spd_handle* h, int32_t top_k, float temperature, const float* uniforms,
                            int32_t positions);

/* Draft-module schedule (Section 3.3's choice against the ablation of Section 4.5). post_step = 0
 * (default): the PDM reads the pre-step features and runs beside the stage compute. post_step = 1:
 * it runs after the step's stage compute on main_stream, before the exit head, and reads every
 * in-flight token one stage deeper (the newest token's anchors 0 and 1 instead of its embedding);
 * drafting is then serial behind the step. Rows recomputed, the draft's position and the verify are
 * unchanged. Legal in any state; SPD_E_INVAL for other values. */
spd_status spd_set_pdm_schedule(spd_handle* h, int32_t post_step);

/* Steps per replayed graph in spd_run_steps (graph mode): `steps` consecutive steps are captured into
 * one graph, so the device runs them with no host launch between them; a remainder below `steps`
 * replays the one-step graph. steps in [1, 16] (default 1); SPD_E_INVAL otherwise. Results are
 * identical for every value. */
spd_status spd_set_graph_steps(spd_handle* h, int32_t steps);

/* Enqueue `count` steps without host synchronisation (needs auto_rollback = 1). If log is not
 * NULL (host, count entries) the call waits and fills it with each step's result; otherwise it
 * returns once the work is enqueued and spd_sync() waits. */
spd_status spd_run_steps(spd_handle* h, int32_t count, spd_step_result* log);

/* Wait for all enqueued work; if last is not NULL store the latest step result there. */
spd_status spd_sync(spd_handle* h, spd_step_result* last);

/* Debug and parity reads (synchronous; host destination). what:
 *   SPD_DBG_RESID:       n*d fp32, in-flight residual streams; position q lives in row q mod n
 *   SPD_DBG_ANCHORS:     n*n*d fp32, [row q mod n][anchor j][d], anchor j = H^{beta_j}
 *   SPD_DBG_PDM_HIDDEN:  8*d fp32, the PDM's output rows of the last step (row i = position c+i)
 *   SPD_DBG_EXIT_LOGITS: V fp32, target logits of the last exiting token (needs spd_set_debug)
 *   SPD_DBG_PDM_LOGITS:  V fp32, the PDM's logits of the last step (needs spd_set_debug)
 *   SPD_DBG_TOKENS:      max_tokens int32, token id per position
 *   SPD_DBG_STATE:       4 int32: c, a, prompt_len, steps
 *   SPD_DBG_KTRACE:      nkslots x 2 uint64 wall-clock stamps of the last step run with
 *                        spd_set_kernel_trace on: per slot the first workgroup's start and the
 *                        latest workgroup end (both 0: nothing ran). Slot (j*5 + k)*n + s
 *                        is sublayer k (QKV, attention, O-proj, gate/up, down) of layer slot j of stage
 *                        s (stage launches); slots 5*J*n + 0, 1, 2 are the LM head,
 *                        verify and the PDM feature projection.
 *   SPD_DBG_QDIST:       sampled decoding: the draft distribution q kept with each in-flight token,
 *                        row r = position mod n: n int32 entry counts, then [n][64] int32 ids, then
 *                        [n][64] fp32 probabilities (value-descending order)
 * bytes must equal the size listed (nkslots from spd_step_plan_info). */
enum {
  SPD_DBG_RESID = 1,
  SPD_DBG_ANCHORS = 2,
  SPD_DBG_PDM_HIDDEN = 3,
  SPD_DBG_EXIT_LOGITS = 4,
  SPD_DBG_PDM_LOGITS = 5,
  SPD_DBG_TOKENS = 6,
  SPD_DBG_STATE = 7,
  SPD_DBG_KTRACE = 10,
  SPD_DBG_QDIST = 11
};
spd_status spd_read_debug(spd_handle* h, int32_t what, void* host, size_t bytes);

/* Copy K and V of positions [pos0, pos0+count) of one layer (pdm = 0: target layer, 1: PDM layer)
 * to host arrays [count x Hkv x dh] in the config's dtype. */
spd_status spd_read_kv(spd_handle* h, int32_t pdm, int32_t layer, int32_t pos0, int32_t count,
                       void* host_k, void* host_v);

/* 1: steps without a per-call draft override replay a HIP graph of the step (both streams, captured
 * on first use) instead of issuing each launch; 0 (default): issue the launches. The step's launch
 * sequence does not depend on host state, so one capture serves every step. */
spd_status spd_set_graph(spd_handle* h, int32_t on);

/* How the stage compute of a step is launched (Section 3.1: every active stage advances its token by
 * one stage). Both modes give bit-identical results (the per-row arithmetic is the same).
 *   mode 0: five launches per layer slot (QKV, attention, O-proj, gate/up, down) on main_stream, each
 *           covering all stages.
 *   mode 2 (default): the stages are spread over `groups` groups of consecutive stages (at most n;
 *           0: the default, 2; -1 keeps the current value); each group runs its own chain of five
 *           launches per layer slot, each covering the group's stages, on its own stream (the
 *           library's, default priority), forked from and joined to main_stream, so that one group's
 *           attention and launch tails can overlap the other groups' weight streaming.
 * `grid` sets the workgroups of one sublayer launch (0: the default): each stages its input vector
 * once and its waves stream their weight rows back to back. SPD_E_INVAL for another mode, a grid
 * above 65535 or groups outside [-1, 8]. */
spd_status spd_set_step_kernel(spd_handle* h, int32_t mode, int32_t grid, int32_t groups);

/* 0: steps skip the Pipeline Draft Module's launches (feature projection and decoder layers; the
 * two-row LM head still runs), for measuring how much of the PDM the stage compute hides; drafts
 * should then come from spd_set_forced_drafts. 1 (default): the PDM runs. */
spd_status spd_set_pdm_enabled(spd_handle* h, int32_t on);

/* Achievable-bandwidth probe (no handle): reads `bytes` (16-byte aligned, at least 16) of device
 * memory at buf with 16-byte non-temporal loads from 2048 workgroups, `reps` times on `stream`
 * after one warm-up pass, and returns the mean time of one pass in *ms. sink: device memory for 2048
 * floats (written). */
spd_status spd_probe_hbm_read(const void* buf, size_t bytes, float* sink, int32_t reps, void* stream, double* ms);

/* Where the Pipeline Draft Module's launches go within a step (it reads only pre-step features, so
 * any placement gives the same results): 0 (default): its own stream, forked from main_stream;
 * 1: main_stream, before the stage compute; 2 and 3 (mode 2 only; otherwise 0): the first stage
 * group's stream, before (2) or after (3) that group's stage launches. SPD_E_INVAL otherwise. */
spd_status spd_set_pdm_placement(spd_handle* h, int32_t place);

/* Workgroups of each of the PDM's GEMV launches in a step (0: the default, 32 per 256 MB of PDM
 * weights). The PDM runs beside the stage compute, so its launches are kept small enough to leave
 * most CUs to the stages while still finishing inside the stage compute. */
spd_status spd_set_pdm_grid(spd_handle* h, int32_t wgs);

/* Launch trace: while on, every step first resets the trace and its stage launches, LM head, verify
 * and PDM projection record their wall-clock start and end in it (SPD_DBG_KTRACE). One store per
 * launch and one device atomic per workgroup that nothing waits for; for measurement only. */
spd_status spd_set_kernel_trace(spd_handle* h, int32_t on);

/* info (host, 8 int32): layer slots J, the wall-clock rate of the launch-trace stamps in kHz, the
 * launch-trace slots (nkslots), the SPD width n, the stage groups in effect (1 in mode 0), the PDM
 * placement, and two zeros. */
spd_status spd_step_plan_info(spd_handle* h, int32_t* info);

/* 1: every LM-head pass also writes its full logits (for SPD_DBG_*_LOGITS). */
spd_status spd_set_debug(spd_handle* h, int32_t on);

/* Kernel timing for roofline measurements. kernel selects one launch class of the stage compute
 * (SPD_K_QKV, SPD_K_ATTN, SPD_K_OPROJ, SPD_K_GATEUP, SPD_K_DOWN; SPD_K_HEAD, the LM-head pass, which
 * with the fused two-row head also runs the step's verify; 0 turns timing off). While on, steps
 * issue their launches (no graph replay) and every launch of that class in layer slot >= first_slot
 * (the exit head counts as the slot after the last) hands two HIP events to its own dispatch, which
 * records the kernel's start and end on the stream it is launched on. A first_slot past the draft
 * module's span times the kernel without the side stream competing for memory bandwidth.
 * spd_kernel_timing waits for the stream, returns the summed kernel time in milliseconds and the
 * number of timed launches, and clears both. */
enum { SPD_K_QKV = 1, SPD_K_ATTN = 2, SPD_K_OPROJ = 3, SPD_K_GATEUP = 4, SPD_K_DOWN = 5, SPD_K_HEAD = 6,
       SPD_K_SPANS = 7 };
spd_status spd_set_kernel_timing(spd_handle* h, int32_t kernel, int32_t first_slot);
spd_status spd_kernel_timing(spd_handle* h, double* total_ms, int32_t* launches);

/* Overlap of the draft module with the stage compute (Section 3.3: drafting must finish within the
 * pipeline step). With spd_set_kernel_timing(h, SPD_K_SPANS) every step records three HIP events: the
 * step's start on main_stream, the end of the PDM's work on pdm_stream, and the end of the stage
 * compute plus exit LM head on main_stream (the point where verification waits for the draft).
 * spd_span_timing waits for both streams and returns, summed over the timed steps: stage_ms (start to
 * end of stage compute), pdm_ms (start to end of the PDM), late_ms (the sum of max(0, pdm end - stage
 * end), i.e. time the verification waited for the draft), and the number of steps; then clears them. */
spd_status spd_span_timing(spd_handle* h, double* stage_ms, double* pdm_ms, double* late_ms, int32_t* steps);

/* Ragged paged decode attention (Section 3.1: every in-flight token attends, at its own position, over
 * the cache of the layer it is on) for up to 8 query rows of one layer, as a call of its own. It runs
 * the step's attention split code: one workgroup per (key split, KV head, row), the last split of a
 * (row, head) to finish merging its splits in split order.
 *   q: device fp32 [nrows][n_q_heads][head_dim], the rows' rotated queries (query head h reads KV
 *      head h / (n_q_heads / n_kv_heads)); scores are scaled by 1/sqrt(head_dim).
 *   kv: device, one layer's pool [num_pages][K, V][n_kv_heads][16 keys][head_dim] of dtype.
 *   page_table: device int32 [num_pages]: logical page i (keys 16i..16i+15) is at physical page
 *      page_table[i], each in [0, num_pages).
 *   lens: host int32 [nrows], row i attends keys [0, lens[i]); 1 <= lens[i] <= 16 * num_pages.
 *   out: device fp32 [nrows][n_q_heads][head_dim].
 *   chunk: keys per split, a positive multiple of 16, with ceil(max lens / chunk) <= 64 splits.
 *   workspace: device, 256-byte aligned, scratch for the split records and tickets: at least
 *      ceil256(4 * nrows * n_kv_heads * splits * 8 * (head_dim + 2)) + 4 * nrows * n_kv_heads bytes.
 * Limits: head_dim 64 or 128; n_q_heads / n_kv_heads in {1, 2, 4, 8}; 1 <= nrows <= 8. The caller owns
 * every buffer. Asynchronous on stream (a hipStream_t). SPD_E_INVAL for other arguments (checked on the
 * host before anything is launched), SPD_E_CAPACITY for a workspace too small, SPD_E_HIP if the launch
 * fails; spd_last_error(NULL) has the message. */
spd_status spd_decode_attention(const float* q, const void* kv, const int32_t* page_table, int32_t num_pages,
                                const int32_t* lens, int32_t nrows, int32_t n_q_heads, int32_t n_kv_heads,
                                int32_t head_dim, int32_t dtype, int32_t chunk, float* out, void* workspace,
                                size_t ws_bytes, void* stream);

/* spd_decode_attention for callers that cannot allocate: code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation. The same arguments and results without the workspace: the
 * split records and tickets live in a static device array of the library, 8.5 MB (2048 split records
 * of head_dim 128, plus 8 KiB of tickets) on each GPU the library runs on, held until the process
 * ends. The call allocates nothing (no hipMalloc, no library allocation); it clears the tickets with a
 * fill kernel before the attention, so a captured call replays correctly. Every call on a GPU uses that
 * GPU's one array and leaves its contents there: calls that overlap on one GPU (other streams, other
 * threads) race, so the caller serializes them. SPD_E_CAPACITY (before anything is launched) when
 * nrows * n_kv_heads * ceil(max lens / chunk) exceeds 2048; otherwise as spd_decode_attention. */
spd_status spd_decode_attention_noalloc(const float* q, const void* kv, const int32_t* page_table,
                                        int32_t num_pages, const int32_t* lens, int32_t nrows, int32_t n_q_heads,
                                        int32_t n_kv_heads, int32_t head_dim, int32_t dtype, int32_t chunk,
                                        float* out, void* stream);

/* Release the handle's events and host buffers (not the caller's memory). NULL is ignored. */
void spd_destroy(spd_handle* h);

const char* spd_status_str(spd_status s);
/* Message of the last failure on this handle ("" if none); NULL handle: last spd_init failure. */
const char* spd_last_error(const spd_handle* h);

#ifdef __cplusplus
}
#endif
#endif /* SPD_H */
