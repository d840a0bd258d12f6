// Persistent step kernel: every layer slot of every active stage of one SPD pipeline step (Section
// 3.1) in one launch.
//
// A step is 5J phases: layer slot j = p / 5 runs the sublayers QKV (+ RMSNorm, RoPE, KV append),
// decode attention, O-proj (+ residual), gate/up (+ RMSNorm, SwiGLU) and down (+ residual, anchor
// capture) for every stage s, stage s on layer beta_s + j. A phase of one stage is a set of tiles;
// phase p of stage s can start once phase p-1 of the same stage has finished, and stages never wait
// for each other (each advances its own token). Workgroups take tickets from one counter and run
// the tiles in the order of a table built on the host, in which every tile comes after the tiles it
// depends on. A workgroup only waits for tiles that lower tickets hold, and those are held by
// workgroups that are already running, so the lowest unfinished ticket can always proceed: the
// launch needs no co-residency and cannot deadlock. Every wait is bounded all the same: on a timeout
// the launch raises a flag (reported by the host as an error) and every later wait returns at once,
// so the grid always drains.
//
// Tiles hand data to each other inside the launch (rotated queries, the new K/V of the token, the
// attention output, the residual stream, the SwiGLU activation). Those values are written with
// device-scope stores and read with device-scope loads, which go to the level every XCD shares; a
// tile's stores complete (s_waitcnt) before it counts itself finished. Weights and the KV written
// by earlier launches are read with ordinary 16-byte loads.
//
// The arithmetic of a row does not depend on how many stages run or which tile order is used: the
// lane-to-column map, the FMA order, the butterfly and the attention split size are fixed, so a
// token's results are identical in an n-stage step and in plain decoding (n = 1).
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>

#include "spd_dev.h"
#include "spd_devfn.h"
#include "spd_gemv.h"
#include "spd_attn.h"

namespace spd {

namespace {


// Trace stamp `which` of a ticket (thread 0; tracing on only).
__device__ __forceinline__ void stamp(const Ctx& C, int ticket, int which) {
  if (C.plan.trace != nullptr && threadIdx.x == 0)
    C.plan.trace[(size_t)ticket * 4 + which] = (unsigned long long)wall_clock64();
}

// All waves' device-scope stores of the tile are complete; count the tile as finished.
__device__ __forceinline__ void finish_tile(int* sync, int idx) {
  wait_own_stores();
  __syncthreads();
  if (threadIdx.x == 0) __hip_atomic_fetch_add(sync + idx, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ------------------------------------------------------------------------------------ step tiles
// One tile of one stage. Each kind is its own function so that the kernel's register budget is the
// largest kind's, not the sum of everything the loop could inline. The context lives in device
// memory (a copy the host keeps current), so passing it costs one pointer.
struct TileArgs {
  int s;           // stage
  int t;           // tile within the (phase, stage)
  int layer;       // beta_s + slot
  int pos;         // the stage's token position
  int dep;         // sync index of the previous phase of this stage (-1: none)
  int dep_target;  // units that phase finishes with
  int done;        // sync index of this tile's phase
  int ticket;
};

// QKV: 16 RoPE pairs (j, j + dh/2) of one q, k or v head; wave w takes pairs 4w .. 4w+3. Applies
// RMSNorm (gain while staging, 1/rms on the dot products), RoPE at the token's own position, and
// appends k, v to the layer's paged cache.
template <typename WT, int DH>
__device__ __noinline__ void tile_qkv(const Ctx* __restrict__ Cp, TileArgs a) {
  extern __shared__ __align__(16) float lds[];
  __shared__ float red[4];
  const Ctx& C = *Cp;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int d = C.d;
  const LayerDesc Ld = C.lay[a.layer];
  const float* x = C.resid + (size_t)(a.pos % C.n) * d;
  constexpr int half = DH / 2, iph = half / kQPairs;
  const int head = a.t / iph, jb = (a.t - head * iph) * kQPairs + w * 4;
  const WT* W;
  int hrow, hk;
  if (head < C.hq) {
    W = (const WT*)Ld.wq;
    hrow = head;
    hk = 0;
  } else if (head < C.hq + C.hkv) {
    W = (const WT*)Ld.wk;
    hrow = head - C.hq;
    hk = 1;
  } else {
    W = (const WT*)Ld.wv;
    hrow = head - C.hq - C.hkv;
    hk = 2;
  }
  const WT* Wh = W + (size_t)(hrow * DH + jb) * d;
  auto rowptr = [&](int rp, int which) { return Wh + (size_t)(rp + which * half) * d; };
  uint4 bA[2][kU], bB[2][kU];
  float r0 = 0.f, r1 = 0.f;
  gemv_prefetch<WT, 4>(rowptr, d, lane, bA, bB);
  if (threadIdx.x == 0 && a.dep >= 0) wait_count(C.plan.sync, a.dep, a.dep_target);
  __syncthreads();  // the inputs are final before any wave loads them
  stamp(C, a.ticket, 1);
  const float ss = stage_vec<Elt<WT>::VE, true>(x, Ld.attn_norm, d, lds, red);
  stamp(C, a.ticket, 2);
  const float sc = 1.0f / sqrtf(ss / (float)d + C.eps);
  gemv_run<WT, 4>(rowptr, d, lane, lds, bA, bB, r0, r1);
  if (lane < 4) {
    const int j = jb + lane;
    float lo = r0 * sc, hi = r1 * sc;
    if (hk != 2) {
      const float2 cs = C.rope[(size_t)a.pos * half + j];
      const float rlo = lo * cs.x - hi * cs.y;
      const float rhi = hi * cs.x + lo * cs.y;
      lo = rlo;
      hi = rhi;
    }
    if (hk == 0) {
      float* qo = C.b[0].q + (size_t)a.s * C.qdim + hrow * DH;
      st_dev(qo + j, lo);
      st_dev(qo + j + half, hi);
    } else {
      WT* kv = (WT*)Ld.kv;
      const size_t off = kv_off(C, a.pos, hrow, j) + (hk == 2 ? (size_t)C.hkv * C.page * DH : 0);
      st_kv_dev<WT>(kv + off, lo);
      st_kv_dev<WT>(kv + off + half, hi);
    }
  }
  finish_tile(C.plan.sync, a.done);
}

template <typename WT, int DH>
__device__ __noinline__ void tile_attn(const Ctx* __restrict__ Cp, TileArgs a) {
  extern __shared__ __align__(16) float lds[];
  const Ctx& C = *Cp;
  const int g = a.t / C.max_splits, split = a.t - g * C.max_splits;
  const int nsplit = (a.pos + C.chunk) / C.chunk;
  if (split >= nsplit) return;
  const int k0 = split * C.chunk, k1 = min(a.pos + 1, k0 + C.chunk);
  const int page0 = C.page_table[min((k0 + (int)threadIdx.x / kAttnTPK) / C.page, C.max_pages - 1)];
  const LayerDesc Ld = C.lay[a.layer];
  if (threadIdx.x == 0) wait_count(C.plan.sync, a.dep, a.dep_target);
  __syncthreads();
  stamp(C, a.ticket, 1);
  const int cidx = a.s * C.hkv + g;
  constexpr int RS = kAttnMaxQ * (DH + 2);
  const bool final_out = attn_split<WT, DH, true>(
      C, (const WT*)Ld.kv, C.b[0].q + (size_t)a.s * C.qdim + g * C.G * DH, C.b[0].ao + (size_t)a.s * C.qdim + g * C.G * DH,
      C.b[0].part + (size_t)cidx * C.max_splits * RS, C.b[0].cnt + cidx, g, split, nsplit, k0, k1, a.pos, page0, lds);
  if (final_out) finish_tile(C.plan.sync, a.done);
}

// O-proj (MODE 0: 16 rows, wave w rows 4w .. 4w+3 in 2 pairs, input = attention output) or down
// (MODE 1: 8 rows, wave w rows 2w, 2w+1, input = SwiGLU activation) with the residual add; down on a
// stage's last layer also keeps the stage output as the next PDM anchor.
template <typename WT, int MODE>
__device__ __noinline__ void tile_proj(const Ctx* __restrict__ Cp, TileArgs a) {
  extern __shared__ __align__(16) float lds[];
  __shared__ float red[4];
  const Ctx& C = *Cp;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int d = C.d, n = C.n;
  const LayerDesc Ld = C.lay[a.layer];
  float* x = C.resid + (size_t)(a.pos % n) * d;
  const int K = MODE == 0 ? C.qdim : C.F;
  const WT* W = (const WT*)(MODE == 0 ? Ld.wo : Ld.wd);
  constexpr int NP = MODE == 0 ? 2 : 1;
  const int m0 = MODE == 0 ? a.t * kORows + w * 4 : a.t * kDRows + w * 2;
  auto rowptr = [&](int rp, int which) {
    const int m = m0 + 2 * rp + which;
    return m < d ? W + (size_t)m * K : (const WT*)nullptr;
  };
  uint4 bA[2][kU], bB[2][kU];
  float r0 = 0.f, r1 = 0.f;
  gemv_prefetch<WT, NP>(rowptr, K, lane, bA, bB);
  if (threadIdx.x == 0) wait_count(C.plan.sync, a.dep, a.dep_target);
  __syncthreads();
  stamp(C, a.ticket, 1);
  stage_vec<Elt<WT>::VE, true>((MODE == 0 ? C.b[0].ao : C.b[0].act) + (size_t)a.s * K, nullptr, K, lds, red);
  stamp(C, a.ticket, 2);
  gemv_run<WT, NP>(rowptr, K, lane, lds, bA, bB, r0, r1);
  float* cap = nullptr;
  if (MODE == 1 && a.layer + 1 == C.beta[a.s + 1] && a.s + 1 <= n - 1)
    cap = C.anchors + ((size_t)(a.pos % n) * n + (a.s + 1)) * d;
  if (lane < NP) {
    const int m = m0 + 2 * lane;
    if (m < d) {
      const float v0 = ld_dev(x + m) + r0;
      st_dev(x + m, v0);
      if (cap != nullptr) cap[m] = v0;
    }
    if (m + 1 < d) {
      const float v1 = ld_dev(x + m + 1) + r1;
      st_dev(x + m + 1, v1);
      if (cap != nullptr) cap[m + 1] = v1;
    }
  }
  finish_tile(C.plan.sync, a.done);
}

// gate/up: 16 outputs, wave w outputs 4w .. 4w+3 with rows (gate m, up m); RMSNorm as in QKV, then
// SwiGLU silu(g) * u.
template <typename WT>
__device__ __noinline__ void tile_gateup(const Ctx* __restrict__ Cp, TileArgs a) {
  extern __shared__ __align__(16) float lds[];
  __shared__ float red[4];
  const Ctx& C = *Cp;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int d = C.d;
  const LayerDesc Ld = C.lay[a.layer];
  const float* x = C.resid + (size_t)(a.pos % C.n) * d;
  const int m0 = a.t * kGOut + w * 4;
  const WT* Wg = (const WT*)Ld.wg;
  const WT* Wu = (const WT*)Ld.wu;
  auto rowptr = [&](int rp, int which) {
    const int m = m0 + rp;
    return m < C.F ? (which ? Wu : Wg) + (size_t)m * d : (const WT*)nullptr;
  };
  uint4 bA[2][kU], bB[2][kU];
  float r0 = 0.f, r1 = 0.f;
  gemv_prefetch<WT, 4>(rowptr, d, lane, bA, bB);
  if (threadIdx.x == 0) wait_count(C.plan.sync, a.dep, a.dep_target);
  __syncthreads();
  stamp(C, a.ticket, 1);
  const float ss = stage_vec<Elt<WT>::VE, true>(x, Ld.mlp_norm, d, lds, red);
  stamp(C, a.ticket, 2);
  const float sc = 1.0f / sqrtf(ss / (float)d + C.eps);
  gemv_run<WT, 4>(rowptr, d, lane, lds, bA, bB, r0, r1);
  if (lane < 4 && m0 + lane < C.F) {
    const float gv = r0 * sc, uv = r1 * sc;
    st_dev(C.b[0].act + (size_t)a.s * C.F + m0 + lane, gv / (1.0f + expf(-gv)) * uv);
  }
  finish_tile(C.plan.sync, a.done);
}

// ------------------------------------------------------------------------------------ step kernel
template <typename WT, int DH>
__global__ __launch_bounds__(kWG, 3) void k_step(const Ctx* __restrict__ Cp) {
  __shared__ int s_ticket;
  const Ctx& C = *Cp;
  int* sync = C.plan.sync;
  const int nitems = C.plan.nitems;
  const int tid = threadIdx.x;
  const int st_a = C.st->a, st_c = C.st->c;  // pre-step state; only the verify kernel changes it
  const int n = C.n;
  if (tid == 0) s_ticket = __hip_atomic_fetch_add(sync + sync_ticket(), 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  __syncthreads();
  for (;;) {
    const int ticket = s_ticket;
    if (ticket >= nitems) break;
    int next = 0;
    if (tid == 0) next = __hip_atomic_fetch_add(sync + sync_ticket(), 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    stamp(C, ticket, 0);
    const uint32_t it = C.plan.items[ticket];
    const int p = (int)(it >> 19), s = (int)((it >> 16) & 7u);
    const int slot = p / 5, kind = p - slot * 5;
    TileArgs a;
    a.s = s;
    a.t = (int)(it & 0xffffu);
    a.layer = C.beta[s] + slot;
    if (s < st_a && a.layer < C.beta[s + 1]) {
      a.pos = st_c + st_a - 1 - s;
      a.dep = p > 0 ? sync_done(p - 1, s, n) : -1;
      a.dep_target = p == 0 ? 0
                     : kind == SK_QKV ? C.plan.tiles[SK_DOWN]
                     : kind == SK_OPROJ ? C.hkv  // attention finishes once per KV head
                                        : C.plan.tiles[kind - 1];
      a.done = sync_done(p, s, n);
      a.ticket = ticket;
      switch (kind) {
        case SK_QKV: tile_qkv<WT, DH>(Cp, a); break;
        case SK_ATTN: tile_attn<WT, DH>(Cp, a); break;
        case SK_OPROJ: tile_proj<WT, 0>(Cp, a); break;
        case SK_GATEUP: tile_gateup<WT>(Cp, a); break;
        default: tile_proj<WT, 1>(Cp, a); break;
      }
    }
    stamp(C, ticket, 3);
    __syncthreads();  // every thread has read s_ticket; LDS free for the next tile
    if (tid == 0) s_ticket = next;
    __syncthreads();
  }
}

}  // namespace

size_t step_lds_bytes(const Ctx& c, int bf16) {
  const int blk = 64 * (bf16 ? 8 : 4);
  int kmax = std::max(std::max(c.d, c.qdim), c.F);
  kmax = (kmax + blk - 1) / blk * blk;
  const size_t gemv = (size_t)kmax * sizeof(float);
  const size_t attn = bf16 ? (c.dh == 128 ? attn_split_lds<uint16_t, 128>() : attn_split_lds<uint16_t, 64>())
                           : (c.dh == 128 ? attn_split_lds<float, 128>() : attn_split_lds<float, 64>());
  return std::max(gemv, attn);
}

void launch_step(const Ctx& c, const Ctx* dev_ctx, int grid, void* stream, int bf16) {
  const size_t shm = step_lds_bytes(c, bf16);
  hipStream_t s = (hipStream_t)stream;
  if (bf16) {
    if (c.dh == 128)
      launch_timed(k_step<uint16_t, 128>, dim3(grid), dim3(kWG), shm, s, dev_ctx);
    else
      launch_timed(k_step<uint16_t, 64>, dim3(grid), dim3(kWG), shm, s, dev_ctx);
  } else {
    if (c.dh == 128)
      launch_timed(k_step<float, 128>, dim3(grid), dim3(kWG), shm, s, dev_ctx);
    else
      launch_timed(k_step<float, 64>, dim3(grid), dim3(kWG), shm, s, dev_ctx);
  }
}

}  // namespace spd
