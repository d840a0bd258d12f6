// gfx950 kernels of one SPD pipeline step.
//
// The step is HBM-bound: each stage multiplies its own layer's weights by one activation vector, so
// every launch below streams weight rows once with 16-byte coalesced loads, keeps activations in
// fp32 (staged in LDS), reduces each row across a 64-lane wavefront in a fixed butterfly order and
// groups all active stages (or all rows of a row block) into one launch per sublayer.
//
// Determinism: a row's result depends only on its weights, its input vector and (for attention) its
// KV length: the lane-to-column map, the FMA order, the butterfly and the split size never depend
// on how many stages share a launch. That makes a token's arithmetic identical whether it runs in an
// n-stage SPD step or in plain decoding (n = 1), which the lossless check relies on.
#include <hip/hip_ext.h>
#include <algorithm>
#include <hip/hip_runtime.h>
#include <math.h>

#include "spd_dev.h"
#include "spd_devfn.h"
#include "spd_gemv.h"
#include "spd_attn.h"
#include "spd_sample.h"

namespace spd {

// ------------------------------------------------------------------------------- row resolution
struct Grp {
  int active;
  int layer;  // target or PDM layer index
  int nrows;
  int pos0;
  int s;      // stage (kind 0) or -1
  int brow0;  // first scratch row of this group
  float* x;   // residual rows: row i at x + i*xstride
  int xstride;
};

__device__ __forceinline__ Grp resolve(const Ctx& C, const Rows& R, int g) {
  Grp r;
  r.active = 1;
  if (R.kind == 0) {
    const int a = C.st->a, c = C.st->c;
    g += R.stage0;
    r.s = g;
    if (g >= a || C.beta[g] + R.slot >= C.beta[g + 1]) {
      r.active = 0;
      return r;
    }
    r.layer = C.beta[g] + R.slot;  // (its weights come from R.ld[g])
    r.nrows = 1;
    r.pos0 = c + a - 1 - g;
    r.brow0 = g;
    r.x = C.resid + (size_t)(r.pos0 % C.n) * C.d;
    r.xstride = C.d;
  } else {
    r.s = -1;
    r.layer = R.layer;
    r.nrows = R.nrows >= 0 ? R.nrows : C.st->a;
    r.pos0 = R.pos0 >= 0 ? R.pos0 : C.st->c;
    r.brow0 = 0;
    r.x = R.x;
    r.xstride = C.d;
    if (r.nrows <= 0) r.active = 0;
  }
  return r;
}

// --------------------------------------------------------------------------------- GEMV building

// Load blocks [blk, min(blk + kU, blk_end)) of every row (block b = columns b*64*VE + lane*VE + 0..VE-1);
// rows that are nullptr or blocks past blk_end load zeros. K is a multiple of VE, so a load that starts
// inside the row ends inside it.
template <typename WT, int RL>
__device__ __forceinline__ void load_blocks(const WT* const (&wr)[RL], int K, int blk, int blk_end, int lane,
                                            uint4 (&w)[RL][kU]) {
  constexpr int VE = Elt<WT>::VE;
  constexpr int BLK = 64 * VE;
#pragma unroll
  for (int u = 0; u < kU; u++) {
#pragma unroll
    for (int r = 0; r < RL; r++) {
      const int col = (blk + u) * BLK + lane * VE;
      w[r][u] = (wr[r] != nullptr && blk + u < blk_end && col < K) ? ldg16(wr[r] + col) : make_uint4(0u, 0u, 0u, 0u);
    }
  }
}

// acc[v][r] += W[row r] . x[v] over staged blocks [0, nbk) of the chunk in LDS (block b of the chunk is
// global block blk0 + b). The first kU blocks must already be in w (prefetched by the caller); later
// groups are loaded here. Per lane the FMA order is: blocks in order, then the VE columns in order.
template <typename WT, int NV, int RL>
__device__ __forceinline__ void accum_blocks(const WT* const (&wr)[RL], int K, int blk0, int nbk, const float* lds,
                                             int KC, int nrows, float (&acc)[NV][RL], uint4 (&w)[RL][kU],
                                             int lane) {
  constexpr int VE = Elt<WT>::VE;
  constexpr int BLK = 64 * VE;
  for (int b = 0; b < nbk; b += kU) {
    if (b > 0) load_blocks<WT, RL>(wr, K, blk0 + b, blk0 + nbk, lane, w);
#pragma unroll
    for (int u = 0; u < kU; u++) {
      if (b + u < nbk) {
        float wf[RL][VE];
#pragma unroll
        for (int r = 0; r < RL; r++) unpack16<WT>(w[r][u], wf[r]);
#pragma unroll
        for (int v = 0; v < NV; v++) {
          if (v < nrows) {
            float x[VE];
            const float* xb = lds + v * KC + (b + u) * BLK;
            const float4 x0 = *reinterpret_cast<const float4*>(xb + lane * 4);
            x[0] = x0.x;
            x[1] = x0.y;
            x[2] = x0.z;
            x[3] = x0.w;
            if constexpr (VE == 8) {
              const float4 x1 = *reinterpret_cast<const float4*>(xb + 256 + lane * 4);
              x[4] = x1.x;
              x[5] = x1.y;
              x[6] = x1.z;
              x[7] = x1.w;
            }
#pragma unroll
            for (int r = 0; r < RL; r++) {
#pragma unroll
              for (int e = 0; e < VE; e++) acc[v][r] = fmaf(wf[r][e], x[e], acc[v][r]);
            }
          }
        }
      }
    }
  }
}

// Source of the activation vectors a GEMV multiplies.
enum XSrc {
  XS_NORM_RESID = 0,  // rmsnorm(residual row) * gain: gain applied while staging, 1/rms at the end
  XS_PLAIN = 1,       // a scratch row, as is
  XS_ANCHORS = 2      // PDM feature input: concatenated eligible anchors, zeros for the rest
};

struct XSpec {
  int src = 0;
  const float* gain[kMaxRows];  // XS_NORM_RESID: gain of row v
  const float* row[kMaxRows];  // activation row v (16-byte aligned)
  int nelig[kMaxRows];         // XS_ANCHORS: eligible length (f+1)*d per row
};

// Stage chunk [kc0, kc0+kl) of every row into LDS (zero padded to kl_pad) with 16-byte loads, all of a
// thread's loads of a round issued before its LDS stores; accumulate the sum of squares per row in ss
// (per-thread partials) when normalising. kl, kc0 and every nelig are multiples of 4.
template <int VE, int NV>
__device__ __forceinline__ void stage_chunk(const XSpec& xs, int nrows, int kc0, int kl, int kl_pad, float* lds,
                                            int KC, float (&ss)[NV]) {
  constexpr int RND = 4;
  const int n4 = kl_pad >> 2;
#pragma unroll
  for (int v = 0; v < NV; v++) {
    if (v >= nrows) continue;
    const float* row = xs.row[v];
    const int nel = xs.src == XS_ANCHORS ? xs.nelig[v] : 0x7fffffff;
    for (int k40 = threadIdx.x; k40 < n4; k40 += kWG * RND) {
      float4 xv[RND], gv[RND];
#pragma unroll
      for (int j = 0; j < RND; j++) {
        const int k = (k40 + j * kWG) * 4;
        const int gk = kc0 + k;
        const bool ok = k < kl && gk < nel;
        xv[j] = ok ? *reinterpret_cast<const float4*>(row + gk) : make_float4(0.f, 0.f, 0.f, 0.f);
        if (xs.src == XS_NORM_RESID)
          gv[j] = ok ? *reinterpret_cast<const float4*>(xs.gain[v] + gk) : make_float4(0.f, 0.f, 0.f, 0.f);
      }
#pragma unroll
      for (int j = 0; j < RND; j++) {
        const int k4 = k40 + j * kWG;
        if (k4 < n4) {
          float4 val = xv[j];
          if (xs.src == XS_NORM_RESID) {
            ss[v] = fmaf(val.x, val.x, ss[v]);
            ss[v] = fmaf(val.y, val.y, ss[v]);
            ss[v] = fmaf(val.z, val.z, ss[v]);
            ss[v] = fmaf(val.w, val.w, ss[v]);
            val.x *= gv[j].x;
            val.y *= gv[j].y;
            val.z *= gv[j].z;
            val.w *= gv[j].w;
          }
          *reinterpret_cast<float4*>(lds + v * KC + xidx<VE>(k4 * 4)) = val;
        }
      }
    }
  }
}


// Staged activation floats per row and chunk (multiples of every block width, so that the
// per-lane accumulation order does not depend on the chunking). LDS stays at 48 KB or less.
constexpr int kChunkCap1 = 12288;
constexpr int kChunkCapN = 1536;

template <int NV>
__device__ __forceinline__ int chunk_floats(int K, int blk) {
  const int kp = (K + blk - 1) / blk * blk;
  const int cap = (NV == 1 ? kChunkCap1 : kChunkCapN);
  return kp < cap ? kp : cap;
}

// One GEMV tile: RL weight rows per wave against NV activation rows. The first weight blocks are
// requested before the activations are staged (they do not depend on them), then every chunk is
// staged and consumed. On return every lane of a wave holds the wave's row results, scaled by 1/rms
// for normalised inputs.
template <typename WT, int NV, int RL>
__device__ __forceinline__ void gemv_tile(const WT* const (&wr)[RL], int K, const XSpec& xs, int nrows,
                                          float eps, float* lds, int KC, float (&acc)[NV][RL]) {
  constexpr int VE = Elt<WT>::VE;
  constexpr int BLK = 64 * VE;
  __shared__ float red[4];
  const int lane = threadIdx.x & 63;
  float ss[NV];
#pragma unroll
  for (int v = 0; v < NV; v++) {
    ss[v] = 0.f;
#pragma unroll
    for (int r = 0; r < RL; r++) acc[v][r] = 0.f;
  }
  uint4 w[RL][kU];
  {
    const int kl0 = min(KC, K);
    load_blocks<WT, RL>(wr, K, 0, (kl0 + BLK - 1) / BLK, lane, w);
  }
  for (int kc0 = 0; kc0 < K; kc0 += KC) {
    const int kl = min(KC, K - kc0);
    const int kl_pad = (kl + BLK - 1) / BLK * BLK;
    const int blk0 = kc0 / BLK, nbk = kl_pad / BLK;
    if (kc0 > 0) {
      __syncthreads();  // every wave is done with the previous chunk
      load_blocks<WT, RL>(wr, K, blk0, blk0 + nbk, lane, w);
    }
    stage_chunk<VE, NV>(xs, nrows, kc0, kl, kl_pad, lds, KC, ss);
    __syncthreads();
    accum_blocks<WT, NV, RL>(wr, K, blk0, nbk, lds, KC, nrows, acc, w, lane);
  }
#pragma unroll
  for (int v = 0; v < NV; v++) {
#pragma unroll
    for (int r = 0; r < RL; r++) acc[v][r] = wave_sum(acc[v][r]);
  }
  if (xs.src == XS_NORM_RESID) {
#pragma unroll
    for (int v = 0; v < NV; v++) {
      const float tot = block_sum(ss[v], red);  // every workgroup reduces in the same order
      const float sc = 1.0f / sqrtf(tot / (float)K + eps);
#pragma unroll
      for (int r = 0; r < RL; r++) acc[v][r] *= sc;
    }
  }
}

enum SKind { SG_QKV = 0, SG_OPROJ = 2, SG_GATEUP = 3, SG_DOWN = 4 };

// Workgroup bx of nbx working on one stage's sublayer (gr: the stage's row, Ld: its layer, set: the
// scratch set). The first weight units are requested before anything the previous sublayer wrote is
// read.
template <typename WT, int KIND>
__device__ __forceinline__ void sgemv_part(const Ctx& C, const Grp& gr, const LayerDesc& Ld, int set, int bx,
                                           int nbx) {
  extern __shared__ __align__(16) float lds[];
  __shared__ float red[4];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int NW = nbx * 4, wv = bx * 4 + w;
  const int d = C.d, dh = C.dh, half = C.dh >> 1;
  const int K = KIND == SG_OPROJ ? C.qdim : (KIND == SG_DOWN ? C.F : d);
  const int npairs = KIND == SG_QKV ? (C.hq + 2 * C.hkv) * half : (KIND == SG_GATEUP ? C.F : (d + 1) / 2);
  const int count = wv < npairs ? (npairs - 1 - wv) / NW + 1 : 0;  // at most 64 (the host sizes the grid)
  const int pos = gr.pos0;
  float* x = gr.x;
  auto rowptr = [&](int i, int which) -> const WT* {
    const int q = wv + i * NW;
    if (KIND == SG_QKV) {
      const int head = q / half, j = q - head * half;
      const WT* W = head < C.hq ? (const WT*)Ld.wq : (head < C.hq + C.hkv ? (const WT*)Ld.wk : (const WT*)Ld.wv);
      const int hrow = head < C.hq ? head : (head < C.hq + C.hkv ? head - C.hq : head - C.hq - C.hkv);
      return W + (size_t)(hrow * dh + j + which * half) * d;
    } else if (KIND == SG_GATEUP) {
      return (which ? (const WT*)Ld.wu : (const WT*)Ld.wg) + (size_t)q * d;
    } else {
      const int m = 2 * q + which;
      const WT* W = (const WT*)(KIND == SG_OPROJ ? Ld.wo : Ld.wd);
      return m < d ? W + (size_t)m * K : (const WT*)nullptr;
    }
  };
  uint4 bA[2][kU], bB[2][kU];
  stream_prefetch<WT>(rowptr, count, K, lane, bA, bB);
  // per-pair values for the epilogue, lane i holding pair i's
  float2 pv = make_float2(0.f, 0.f);
  int page = 0;
  if (KIND == SG_QKV) {
    if (lane < count) {
      const int q = wv + lane * NW, j = q % half;
      pv = C.rope[(size_t)pos * half + j];
    }
    page = C.page_table[pos / C.page];
  }
  if (KIND == SG_OPROJ || KIND == SG_DOWN) {
    if (lane < count) {
      const int m = 2 * (wv + lane * NW);
      pv.x = x[m];
      pv.y = m + 1 < d ? x[m + 1] : 0.f;
    }
  }
  float sc = 1.f;
  if (KIND == SG_QKV || KIND == SG_GATEUP) {
    const float ss = stage_vec<Elt<WT>::VE>(x, KIND == SG_QKV ? Ld.attn_norm : Ld.mlp_norm, d, lds, red);
    sc = 1.0f / sqrtf(ss / (float)d + C.eps);
  } else {
    stage_vec<Elt<WT>::VE>((KIND == SG_OPROJ ? C.b[set].ao : C.b[set].act) + (size_t)gr.brow0 * K,
                                nullptr, K, lds, red);
  }
  float* cap = nullptr;
  if (KIND == SG_DOWN && gr.layer + 1 == C.beta[gr.s + 1] && gr.s + 1 <= C.n - 1)
    cap = C.anchors + ((size_t)(pos % C.n) * C.n + (gr.s + 1)) * d;
  auto done = [&](int i, float s0, float s1) {
    const float2 v = make_float2(__shfl(pv.x, i, 64), __shfl(pv.y, i, 64));
    if (lane != 0) return;
    const int q = wv + i * NW;
    if (KIND == SG_QKV) {
      const int head = q / half, j = q - head * half;
      float lo = s0 * sc, hi = s1 * sc;
      if (head < C.hq + C.hkv) {  // q and k are rotated at the token's own position
        const float rlo = lo * v.x - hi * v.y;
        const float rhi = hi * v.x + lo * v.y;
        lo = rlo;
        hi = rhi;
      }
      if (head < C.hq) {
        float* qo = C.b[set].q + (size_t)gr.brow0 * C.qdim + head * dh;
        qo[j] = lo;
        qo[j + half] = hi;
      } else {
        const int hk = head < C.hq + C.hkv ? head - C.hq : head - C.hq - C.hkv;
        WT* kv = (WT*)Ld.kv;
        const size_t off = (size_t)page * (2 * C.hkv * C.page * dh) + ((size_t)hk * C.page + (pos % C.page)) * dh + j +
                           (head < C.hq + C.hkv ? 0 : (size_t)C.hkv * C.page * dh);
        st1<WT>(kv, off, lo);
        st1<WT>(kv, off + half, hi);
      }
    } else if (KIND == SG_GATEUP) {
      const float g = s0 * sc, u = s1 * sc;
      float* ao = C.b[set].act + (size_t)gr.brow0 * C.F + q;
      *ao = g / (1.0f + expf(-g)) * u;
    } else {
      const int m = 2 * q;
      const float n0 = v.x + s0;
      x[m] = n0;
      if (cap != nullptr) cap[m] = n0;
      if (m + 1 < d) {
        const float n1 = v.y + s1;
        x[m + 1] = n1;
        if (cap != nullptr) cap[m + 1] = n1;
      }
    }
  };
  stream_run<WT>(rowptr, done, count, K, lane, lds, bA, bB);
}

template <typename WT, int KIND>
__global__ __launch_bounds__(kWG) void k_sgemv(Ctx C, Rows R) {
  const Grp gr = resolve(C, R, blockIdx.y);
  if (!gr.active) return;
  const int ts = ktrace_slot(C, R.slot, KIND, gr.s);
  ktrace_start(C, ts, blockIdx.x == 0);
  sgemv_part<WT, KIND>(C, gr, R.ld[gr.s], R.set, blockIdx.x, gridDim.x);  // stage launches carry their layers
  ktrace_end(C, ts);
}

// ----------------------------------------------------------- row-block streaming GEMVs (PDM)
// A sublayer of a row block whose rows all use the same layer (the PDM's decoder layer over its a
// rows, row i at position pos0 + i): the weights are streamed as in the stage launches, but every
// pair is applied to up to nrp rows staged together in LDS (nrp fits the rows' input vectors in the
// workgroup's LDS; more rows take further passes over the weights). Epilogues as in sgemv_part, row
// r's handled by lane r: QKV rotates at the row's position and appends K/V to the layer's cache,
// O-proj and down add into the row's residual stream, gate/up applies SwiGLU.
template <typename WT, int KIND, int NR>
__global__ __launch_bounds__(kWG) void k_rgemv(Ctx C, Rows R, int nrp) {
  extern __shared__ __align__(16) float lds[];
  __shared__ float red[4];
  const Grp gr = resolve(C, R, 0);
  if (!gr.active) return;
  const LayerDesc Ld = C.lay[gr.layer];
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int NW = gridDim.x * 4, wv = blockIdx.x * 4 + w;
  const int d = C.d, dh = C.dh, half = C.dh >> 1;
  constexpr int BLK = 64 * Elt<WT>::VE;
  const int K = KIND == SG_OPROJ ? C.qdim : (KIND == SG_DOWN ? C.F : d);
  const int ldsK = (K + BLK - 1) / BLK * BLK;
  const int npairs = KIND == SG_QKV ? (C.hq + 2 * C.hkv) * half : (KIND == SG_GATEUP ? C.F : (d + 1) / 2);
  const int count = wv < npairs ? (npairs - 1 - wv) / NW + 1 : 0;  // at most 64 (the host sizes the grid)
  auto rowptr = [&](int i, int which) -> const WT* {
    const int q = wv + i * NW;
    if (KIND == SG_QKV) {
      const int head = q / half, j = q - head * half;
      const WT* W = head < C.hq ? (const WT*)Ld.wq : (head < C.hq + C.hkv ? (const WT*)Ld.wk : (const WT*)Ld.wv);
      const int hrow = head < C.hq ? head : (head < C.hq + C.hkv ? head - C.hq : head - C.hq - C.hkv);
      return W + (size_t)(hrow * dh + j + which * half) * d;
    } else if (KIND == SG_GATEUP) {
      return (which ? (const WT*)Ld.wu : (const WT*)Ld.wg) + (size_t)q * d;
    } else {
      const int m = 2 * q + which;
      const WT* W = (const WT*)(KIND == SG_OPROJ ? Ld.wo : Ld.wd);
      return m < d ? W + (size_t)m * K : (const WT*)nullptr;
    }
  };
  for (int r0 = 0; r0 < gr.nrows; r0 += nrp) {
    const int nr = min(nrp, gr.nrows - r0);
    if (r0 > 0) __syncthreads();  // every wave is done with the previous rows' vectors
    uint4 bA[2][kU], bB[2][kU];
    stream_prefetch<WT>(rowptr, count, K, lane, bA, bB);
    // per-pair epilogue values of every row, lane i holding pair i's
    float2 pv[NR];
    int page[NR];
#pragma unroll
    for (int r = 0; r < NR; r++) {
      pv[r] = make_float2(0.f, 0.f);
      page[r] = 0;
      if (r < nr) {
        const int pos = gr.pos0 + r0 + r;
        const float* xr = gr.x + (size_t)(r0 + r) * gr.xstride;
        if (KIND == SG_QKV) {
          if (lane < count) pv[r] = C.rope[(size_t)pos * half + (wv + lane * NW) % half];
          page[r] = C.page_table[pos / C.page];
        } else if (KIND == SG_OPROJ || KIND == SG_DOWN) {
          if (lane < count) {
            const int m = 2 * (wv + lane * NW);
            pv[r].x = xr[m];
            pv[r].y = m + 1 < d ? xr[m + 1] : 0.f;
          }
        }
      }
    }
    float sc[NR];
#pragma unroll
    for (int r = 0; r < NR; r++) {
      sc[r] = 1.f;
      if (r < nr) {
        if (KIND == SG_QKV || KIND == SG_GATEUP) {
          const float ss = stage_vec<Elt<WT>::VE>(gr.x + (size_t)(r0 + r) * gr.xstride,
                                                          KIND == SG_QKV ? Ld.attn_norm : Ld.mlp_norm, d,
                                                          lds + (size_t)r * ldsK, red);
          sc[r] = 1.0f / sqrtf(ss / (float)d + C.eps);
        } else {
          stage_vec<Elt<WT>::VE>((KIND == SG_OPROJ ? C.b[R.set].ao : C.b[R.set].act) +
                                            (size_t)(gr.brow0 + r0 + r) * K,
                                        nullptr, K, lds + (size_t)r * ldsK, red);
        }
      }
    }
    // down of a prefill row block ending a stage: its output is also that stage's anchor of the row
    float* cap = (KIND == SG_DOWN && R.anch != nullptr && R.cap >= 0) ? R.anch + (size_t)R.cap * d : nullptr;
    auto done = [&](int i, const float (&s0)[NR], const float (&s1)[NR]) {
      float2 v[NR];
#pragma unroll
      for (int r = 0; r < NR; r++) v[r] = make_float2(__shfl(pv[r].x, i, 64), __shfl(pv[r].y, i, 64));
      const int q = wv + i * NW;
#pragma unroll
      for (int r = 0; r < NR; r++) {
        if (lane != r || r >= nr) continue;
        const int row = r0 + r, pos = gr.pos0 + row;
        if (KIND == SG_QKV) {
          const int head = q / half, j = q - head * half;
          float lo = s0[r] * sc[r], hi = s1[r] * sc[r];
          if (head < C.hq + C.hkv) {
            const float rlo = lo * v[r].x - hi * v[r].y;
            const float rhi = hi * v[r].x + lo * v[r].y;
            lo = rlo;
            hi = rhi;
          }
          if (head < C.hq) {
            float* qo = C.b[R.set].q + (size_t)(gr.brow0 + row) * C.qdim + head * dh;
            qo[j] = lo;
            qo[j + half] = hi;
          } else {
            const int hk = head < C.hq + C.hkv ? head - C.hq : head - C.hq - C.hkv;
            WT* kv = (WT*)Ld.kv;
            const size_t off = (size_t)page[r] * (2 * C.hkv * C.page * dh) +
                               ((size_t)hk * C.page + (pos % C.page)) * dh + j +
                               (head < C.hq + C.hkv ? 0 : (size_t)C.hkv * C.page * dh);
            st1<WT>(kv, off, lo);
            st1<WT>(kv, off + half, hi);
          }
        } else if (KIND == SG_GATEUP) {
          const float g = s0[r] * sc[r], u = s1[r] * sc[r];
          C.b[R.set].act[(size_t)(gr.brow0 + row) * C.F + q] = g / (1.0f + expf(-g)) * u;
        } else {
          const int m = 2 * q;
          float* xr = gr.x + (size_t)row * gr.xstride;
          const float n0 = v[r].x + s0[r], n1 = v[r].y + s1[r];
          xr[m] = n0;
          if (m + 1 < d) xr[m + 1] = n1;
          if (cap != nullptr) {
            float* cr = cap + (size_t)row * C.n * d;
            cr[m] = n0;
            if (m + 1 < d) cr[m + 1] = n1;
          }
        }
      }
    };
    rstream_run<WT, NR>(rowptr, done, count, K, lane, lds, ldsK, nr, bA, bB);
  }
}

// K-split row-block GEMV: the same sublayers as k_rgemv, for row blocks whose input vectors do not fit
// the LDS budget at full width. Workgroup (x, y) stages chunk y (kRowSplitK inputs) of every row and
// streams its pairs over that chunk only, in the same per-wave FMA order as k_rgemv, so each weight is
// read once and the workgroup holds a small LDS slice, leaving room on its compute unit for other work.
// Each chunk's dot products (and, for the normed sublayers, its sums of squares) go to split records;
// the workgroup of column x that finishes last (a ticket per column, zero at rest) adds the chunks in
// chunk order and runs the epilogue of the column's pairs, then resets the ticket.
// Records: pair q of row r, chunk y at part[((y * kMaxRows + r) * npairs + q) * 2]; the sums of
// squares of column x after them, at [(x * chunks + y) * kMaxRows + r].
template <typename WT, int KIND, int NR>
__global__ __launch_bounds__(kWG) void k_rgemv_ks(Ctx C, Rows R) {
  extern __shared__ __align__(16) float lds[];
  __shared__ float red[4];
  __shared__ float s_sc[kMaxRows];
  __shared__ int s_last;
  const Grp gr = resolve(C, R, 0);
  if (!gr.active) return;
  const LayerDesc Ld = C.lay[gr.layer];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int NW = gridDim.x * 4, wv = blockIdx.x * 4 + w;
  const int d = C.d, dh = C.dh, half = C.dh >> 1;
  const int K = KIND == SG_OPROJ ? C.qdim : (KIND == SG_DOWN ? C.F : d);
  const int ns = gridDim.y, y = blockIdx.y;
  const int k0 = y * kRowSplitK, KC = min(kRowSplitK, K - k0);
  const int npairs = KIND == SG_QKV ? (C.hq + 2 * C.hkv) * half : (KIND == SG_GATEUP ? C.F : (d + 1) / 2);
  const int count = wv < npairs ? (npairs - 1 - wv) / NW + 1 : 0;  // at most 64 (the host sizes the grid)
  const int nr = gr.nrows;                                          // at most NR (the host checks)
  constexpr bool NORM = KIND == SG_QKV || KIND == SG_GATEUP;
  float* part = C.b[R.set].rpart;
  float* ssq = part + (size_t)ns * kMaxRows * npairs * 2;
  auto rowptr = [&](int i, int which) -> const WT* {
    const int q = wv + i * NW;
    const WT* p;
    if (KIND == SG_QKV) {
      const int head = q / half, j = q - head * half;
      const WT* W = head < C.hq ? (const WT*)Ld.wq : (head < C.hq + C.hkv ? (const WT*)Ld.wk : (const WT*)Ld.wv);
      const int hrow = head < C.hq ? head : (head < C.hq + C.hkv ? head - C.hq : head - C.hq - C.hkv);
      p = W + (size_t)(hrow * dh + j + which * half) * d;
    } else if (KIND == SG_GATEUP) {
      p = (which ? (const WT*)Ld.wu : (const WT*)Ld.wg) + (size_t)q * d;
    } else {
      const int m = 2 * q + which;
      if (m >= d) return (const WT*)nullptr;
      p = (const WT*)(KIND == SG_OPROJ ? Ld.wo : Ld.wd) + (size_t)m * K;
    }
    return p + k0;
  };
  uint4 bA[2][kU], bB[2][kU];
  stream_prefetch<WT>(rowptr, count, KC, lane, bA, bB);
  float ss[NR];
#pragma unroll
  for (int r = 0; r < NR; r++) {
    ss[r] = 0.f;
    if (r < nr) {
      if (NORM)
        ss[r] = stage_vec<Elt<WT>::VE>(gr.x + (size_t)r * gr.xstride + k0,
                                       (KIND == SG_QKV ? Ld.attn_norm : Ld.mlp_norm) + k0, KC,
                                       lds + (size_t)r * kRowSplitK, red);
      else
        stage_vec<Elt<WT>::VE>((KIND == SG_OPROJ ? C.b[R.set].ao : C.b[R.set].act) + (size_t)(gr.brow0 + r) * K + k0,
                               nullptr, KC, lds + (size_t)r * kRowSplitK, red);
    }
  }
  auto keep = [&](int i, const float (&s0)[NR], const float (&s1)[NR]) {
    const int q = wv + i * NW;
#pragma unroll
    for (int r = 0; r < NR; r++)
      if (lane == r && r < nr) st_dev2f(part + (((size_t)y * kMaxRows + r) * npairs + q) * 2, s0[r], s1[r]);
  };
  rstream_run<WT, NR>(rowptr, keep, count, KC, lane, lds, kRowSplitK, nr, bA, bB);
  if (NORM && tid < nr) {
#pragma unroll
    for (int r = 0; r < NR; r++)
      if (tid == r) st_dev(ssq + ((size_t)blockIdx.x * ns + y) * kMaxRows + r, ss[r]);
  }
  wait_own_stores();
  __syncthreads();
  if (tid == 0) {
    const int t = __hip_atomic_fetch_add(C.b[R.set].rtick + blockIdx.x, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (t == ns - 1);
  }
  __syncthreads();
  if (!s_last) return;
  // the column's last workgroup: the rows' RMSNorm scales, then every (pair, row) of the column
  if (tid < kMaxRows) {
    float sc = 1.f;
    if (NORM && tid < nr) {
      float t = 0.f;
      for (int yy = 0; yy < ns; yy++) t += ld_dev(ssq + ((size_t)blockIdx.x * ns + yy) * kMaxRows + tid);
      sc = 1.0f / sqrtf(t / (float)d + C.eps);
    }
    s_sc[tid] = sc;
  }
  __syncthreads();
  float* cap = (KIND == SG_DOWN && R.anch != nullptr && R.cap >= 0) ? R.anch + (size_t)R.cap * d : nullptr;
  for (int e = lane; e < count * nr; e += 64) {
    const int i = e / nr, r = e - i * nr;
    const int q = wv + i * NW;
    float s0 = 0.f, s1 = 0.f;
    for (int yy = 0; yy < ns; yy++) {
      const float2 v = ld_dev2(part + (((size_t)yy * kMaxRows + r) * npairs + q) * 2);
      s0 += v.x;
      s1 += v.y;
    }
    const float sc = s_sc[r];
    const int pos = gr.pos0 + r;
    if (KIND == SG_QKV) {
      const int head = q / half, j = q - head * half;
      float lo = s0 * sc, hi = s1 * sc;
      if (head < C.hq + C.hkv) {
        const float2 v = C.rope[(size_t)pos * half + j];
        const float rlo = lo * v.x - hi * v.y;
        const float rhi = hi * v.x + lo * v.y;
        lo = rlo;
        hi = rhi;
      }
      if (head < C.hq) {
        float* qo = C.b[R.set].q + (size_t)(gr.brow0 + r) * C.qdim + head * dh;
        qo[j] = lo;
        qo[j + half] = hi;
      } else {
        const int hk = head < C.hq + C.hkv ? head - C.hq : head - C.hq - C.hkv;
        WT* kv = (WT*)Ld.kv;
        const int page = C.page_table[pos / C.page];
        const size_t off = (size_t)page * (2 * C.hkv * C.page * dh) + ((size_t)hk * C.page + (pos % C.page)) * dh + j +
                           (head < C.hq + C.hkv ? 0 : (size_t)C.hkv * C.page * dh);
        st1<WT>(kv, off, lo);
        st1<WT>(kv, off + half, hi);
      }
    } else if (KIND == SG_GATEUP) {
      const float g = s0 * sc, u = s1 * sc;
      C.b[R.set].act[(size_t)(gr.brow0 + r) * C.F + q] = g / (1.0f + expf(-g)) * u;
    } else {
      const int m = 2 * q;
      float* xr = gr.x + (size_t)r * gr.xstride;
      const float n0 = xr[m] + s0;
      const float n1 = m + 1 < d ? xr[m + 1] + s1 : 0.f;
      xr[m] = n0;
      if (m + 1 < d) xr[m + 1] = n1;
      if (cap != nullptr) {
        float* cr = cap + (size_t)r * C.n * d;
        cr[m] = n0;
        if (m + 1 < d) cr[m + 1] = n1;
      }
    }
  }
  if (tid == 0) __hip_atomic_store(C.b[R.set].rtick + blockIdx.x, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// ---------------------------------------------------------------------- PDM feature projection
// g_q = W_in . [H^{beta_0}; ...; H^{beta_f}; 0 ...] for the rows the PDM runs (Eq. agg-main with
// one projection whose column block j serves anchor j). prefill = 1: rows of the prefill chunk
// at full depth; else the a in-flight rows, row i at depth a-1-i. Tile = 8 outputs (2 per wave).
template <typename WT>
__device__ __forceinline__ void pdm_fc_body(const Ctx& C, int prefill, int nrows_arg) {
  extern __shared__ __align__(16) float lds[];
  constexpr int NV = kMaxRows;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int K = C.n * C.d;
  int nrows;
  XSpec xs;
  xs.src = XS_ANCHORS;
  if (prefill) {
    nrows = nrows_arg;
    for (int i = 0; i < kMaxRows; i++) {
      xs.row[i] = C.pf_anch + (size_t)i * C.n * C.d;
      xs.nelig[i] = K;
    }
  } else {
    const int c = C.st->c, a = C.st->a;
    nrows = a;
    for (int i = 0; i < kMaxRows; i++) {
      // in-flight position c+i keeps its anchors in ring row (c+i) mod n
      xs.row[i] = C.anchors + (size_t)((c + i) % C.n) * C.n * C.d;
      // pre-step depth a - 1 - i; the post-step schedule runs after the stage compute, one deeper
      const int depth = a - 1 - i + C.post_step;
      const int f = depth < C.n - 1 ? depth : C.n - 1;
      xs.nelig[i] = (f + 1) * C.d;
    }
  }
  if (nrows <= 0) return;
  const int m0 = blockIdx.x * 8 + w * 2;
  const WT* W = (const WT*)C.w_in;
  const WT* wr[2];
#pragma unroll
  for (int r = 0; r < 2; r++) wr[r] = (m0 + r < C.d) ? W + (size_t)(m0 + r) * K : nullptr;
  const int KC = chunk_floats<NV>(K, 64 * Elt<WT>::VE);
  float acc[NV][2];
  gemv_tile<WT, NV, 2>(wr, K, xs, nrows, 0.f, lds, KC, acc);
  float* out = C.pdm_x;
#pragma unroll
  for (int v = 0; v < NV; v++) {
#pragma unroll
    for (int r = 0; r < 2; r++) {
      if (lane == v * 2 + r && v < nrows && m0 + r < C.d) out[(size_t)v * C.d + m0 + r] = acc[v][r];
    }
  }
}

template <typename WT>
__global__ __launch_bounds__(kWG) void k_pdm_fc(Ctx C, int prefill, int nrows_arg) {
  ktrace_start(C, ktrace_extra(C, KT_PDM), blockIdx.x == 0 && blockIdx.y == 0);
  pdm_fc_body<WT>(C, prefill, nrows_arg);
  ktrace_end(C, ktrace_extra(C, KT_PDM));
}

// ---------------------------------------------------------------------------- LM head + argmax
// Each workgroup folds its best (value, index), the lowest index winning ties, into a 64-bit key
// with a device-scope maximum; the single-workgroup kernel that follows on the stream reads it. The
// (value desc, index asc) order is total, so the winner does not depend on the order of arrival.

// Rows of one LM-head pass. src 0: the exit row (skipped unless a == n); 1: the PDM's last row;
// 2: prefill row `row`; 3: the exit row and the PDM's last row together (rows 0 and 1), one pass over
// W_lm serving both heads. The vocabulary is streamed like a stage GEMV (each workgroup stages the
// normalised rows once, its waves stream vocabulary row pairs back to back); each row's argmax goes
// to the argmax key of set 0 (target) or set 1 (PDM) as an order-independent maximum.
// SAMP: sampled decoding; every logit also goes to the wave's region of C.sam.wlog and the
// workgroup's best key per row to C.sam.wgmax (device-scope stores, read by the launch's last
// workgroup). The logits gather in LDS after the staged rows (lcap floats per wave and row) while
// the vocabulary streams, and each wave writes its region out once at the end, so that no store
// sits between the weight loads; a region over lcap floats is stored as it is produced.
template <typename WT, int NV, bool SAMP = false>
__device__ __forceinline__ void head_body(const Ctx& C, int src, int row, int lcap = 0) {
  extern __shared__ __align__(16) float lds[];
  __shared__ float red[4];
  __shared__ float s_v[NV][4];
  __shared__ int s_i[NV][4];
  const int a = C.st->a, c = C.st->c;
  const float* xr[NV];
  const float* gn[NV];
  int set[NV];
  if (src == 0) {
    if (a != C.n) return;  // nothing exits while the pipeline fills
    xr[0] = C.resid + (size_t)(c % C.n) * C.d;
    gn[0] = C.final_norm;
    set[0] = 0;
  } else if (src == 1) {
    xr[0] = C.pdm_x + (size_t)(a - 1) * C.d;
    gn[0] = C.pdm_norm;
    set[0] = 1;
  } else if (src == 2) {
    xr[0] = C.pf_x + (size_t)row * C.d;
    gn[0] = C.final_norm;
    set[0] = 0;
  } else {
    // while the pipeline fills the exit row is computed but unused (its argmax is not read)
    xr[0] = C.resid + (size_t)(c % C.n) * C.d;
    gn[0] = C.final_norm;
    set[0] = 0;
    xr[NV - 1] = C.pdm_x + (size_t)(a - 1) * C.d;
    gn[NV - 1] = C.pdm_norm;
    set[NV - 1] = 1;
  }
  constexpr int BLK = 64 * Elt<WT>::VE;
  // the PDM's row alone (src 1) goes through its own head when it has one; V counts that head's rows
  const bool own = src == 1 && C.pdm_V > 0;
  const int d = C.d, V = own ? C.pdm_V : C.V;
  const int ldsK = (d + BLK - 1) / BLK * BLK;
  const int w = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int NW = gridDim.x * 4, wv = blockIdx.x * 4 + w;
  const int npairs = (V + 1) / 2;
  const int count = wv < npairs ? (npairs - 1 - wv) / NW + 1 : 0;
  const WT* W = (const WT*)(own ? C.pdm_head : C.lm_head);
  auto rowptr = [&](int i, int which) -> const WT* {
    const int m = 2 * (wv + i * NW) + which;
    return m < V ? W + (size_t)m * d : (const WT*)nullptr;
  };
  uint4 bA[2][kU], bB[2][kU];
  stream_prefetch<WT>(rowptr, count, d, lane, bA, bB);  // weights first, then the rows
  float scl[NV];
#pragma unroll
  for (int v = 0; v < NV; v++) {
    const float ss = stage_vec<Elt<WT>::VE>(xr[v], gn[v], d, lds + (size_t)v * ldsK, red);
    scl[v] = 1.0f / sqrtf(ss / (float)d + C.eps);
  }
  float bv[NV];
  int bi[NV];
#pragma unroll
  for (int v = 0; v < NV; v++) {
    bv[v] = -INFINITY;
    bi[v] = 0x7fffffff;
  }
  const bool dbg_row0 = C.debug && (src != 0 && src != 3 ? true : a == C.n);
  const int cmax = 2 * ((npairs + NW - 1) / NW);  // SAMP: floats per wave region
  const bool lbuf = SAMP && cmax <= lcap;
  float* lg = lds + (size_t)NV * ldsK + (size_t)w * NV * lcap;  // lbuf: [NV][lcap] of this wave
  // every lane holds the same sums, so every lane keeps the same running maximum
  auto done = [&](int i, const float (&s0)[NV], const float (&s1)[NV]) {
    const int m = 2 * (wv + i * NW);
#pragma unroll
    for (int v = 0; v < NV; v++) {
      const float l0 = s0[v] * scl[v], l1 = s1[v] * scl[v];
      if (C.debug && (v > 0 || dbg_row0) && lane < 2 && m + lane < V)
        C.dbg_logits[(size_t)set[v] * C.V + m + lane] = lane == 0 ? l0 : l1;
      if (SAMP && lane < 2 && m + lane < V) {
        if (lbuf)
          lg[v * lcap + 2 * i + lane] = lane == 0 ? l0 : l1;
        else
          st_dev(C.sam.wlog + (size_t)set[v] * C.sam.wlog_stride + (size_t)wv * cmax + 2 * i + lane,
                 lane == 0 ? l0 : l1);
      }
      if (m < V && better(l0, m, bv[v], bi[v])) {
        bv[v] = l0;
        bi[v] = m;
      }
      if (m + 1 < V && better(l1, m + 1, bv[v], bi[v])) {
        bv[v] = l1;
        bi[v] = m + 1;
      }
    }
  };
  rstream_run<WT, NV>(rowptr, done, count, d, lane, lds, ldsK, NV, bA, bB);
  if (lbuf) {  // the wave reads back only what its own lanes wrote (in order within the wave)
#pragma unroll
    for (int v = 0; v < NV; v++)
      for (int e = lane; e < 2 * count; e += 64)
        if (2 * (wv + (e >> 1) * NW) + (e & 1) < V)
          st_dev(C.sam.wlog + (size_t)set[v] * C.sam.wlog_stride + (size_t)wv * cmax + e, lg[v * lcap + e]);
  }
  if (lane == 0) {
#pragma unroll
    for (int v = 0; v < NV; v++) {
      s_v[v][w] = bv[v];
      s_i[v][w] = bi[v];
    }
  }
  __syncthreads();
  if (threadIdx.x < NV) {
    const int v = threadIdx.x;
    float fv = s_v[v][0];
    int fi = s_i[v][0];
    for (int k = 1; k < 4; k++)
      if (better(s_v[v][k], s_i[v][k], fv, fi)) {
        fv = s_v[v][k];
        fi = s_i[v][k];
      }
    // the maximum is order-independent, so the result does not depend on which workgroup lands last
    if (fi != 0x7fffffff)
      __hip_atomic_fetch_max(C.b[set[v]].hkey, argmax_key(fv, fi), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (SAMP)
      __hip_atomic_store(C.sam.wgmax + (size_t)set[v] * kSampleWGs + blockIdx.x,
                         fi != 0x7fffffff ? argmax_key(fv, fi) : 0ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  }
}

template <typename WT, int NV>
__global__ __launch_bounds__(kWG) void k_head(Ctx C, int src, int row) {
  ktrace_start(C, ktrace_extra(C, KT_HEAD), blockIdx.x == 0 && blockIdx.y == 0);
  head_body<WT, NV>(C, src, row);
  ktrace_end(C, ktrace_extra(C, KT_HEAD));
}

// The LM-head argmax of one stream's row, read (and reset to zero for the next pass) by the single
// workgroup that follows the head on the stream.
__device__ __forceinline__ int take_head(const BufSet& B, int V) {
  return argmax_index(*B.hkey, V);
}
// The same, when the key was folded in by other workgroups of the same launch (device-scope load).
__device__ __forceinline__ int take_head_dev(const BufSet& B, int V) {
  return argmax_index(__hip_atomic_load(B.hkey, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT), V);
}
// Rows of the PDM's head, and the target token of its argmax (a draft id with an own head).
__device__ __forceinline__ int pdm_rows(const Ctx& C) { return C.pdm_V > 0 ? C.pdm_V : C.V; }
__device__ __forceinline__ int pdm_token(const Ctx& C, int i) { return C.pdm_V > 0 ? C.pdm_map[i] : i; }

// ------------------------------------------------------------------------------- attention
// Decode attention of a stage launch. Grid: x = key split, y = KV head, z = stage of the launch.
// The page of this thread's first key and the device state are requested together at entry; the
// split itself is attn_split (shared with the persistent step kernel).
// GP: head slots of the split (4 or 8), or 0 to choose from C.G at run time.
template <typename KVT, int DH, int GP = 0>
__device__ __forceinline__ void attn_part(const Ctx& C, int s, int slot, const KVT* kv, int set, int g, int split) {
  extern __shared__ __align__(16) float lds[];
  const int k0 = split * C.chunk;
  const int page0 = C.page_table[min((k0 + (int)threadIdx.x / kAttnTPK) / C.page, C.max_pages - 1)];
  const int st_a = C.st->a, st_c = C.st->c;
  const int layer = C.beta[s] + slot;
  if (s >= st_a || layer >= C.beta[s + 1]) return;  // stage idle in this slot
  const int pos0 = st_c + st_a - 1 - s;             // the stage's token; it attends to keys [0, pos0]
  const int nsplit = (pos0 + C.chunk) / C.chunk;
  if (split >= nsplit) return;
  const int k1 = min(pos0 + 1, k0 + C.chunk);
  const BufSet& B = C.b[set];
  const int cidx = s * C.hkv + g;
  constexpr int RS = kAttnMaxQ * (DH + 2);
  const float* q = B.q + (size_t)s * C.qdim + g * C.G * DH;
  float* out = B.ao + (size_t)s * C.qdim + g * C.G * DH;
  float* rec = B.part + (size_t)cidx * C.max_splits * RS;
  if constexpr (GP == 0)
    attn_split<KVT, DH>(C, kv, q, out, rec, B.cnt + cidx, g, split, nsplit, k0, k1, pos0, page0, lds);
  else
    attn_split_g<KVT, DH, GP>(C, kv, q, out, rec, B.cnt + cidx, g, split, nsplit, k0, k1, pos0, page0, lds);
}

// The stage launch is instantiated per head-slot count, so its registers are those of one variant.
template <typename KVT, int DH, int GP>
__global__ __launch_bounds__(kWG) void k_attn_stage(Ctx C, Rows R) {
  const int s = R.stage0 + blockIdx.z;
  const int ts = ktrace_slot(C, R.slot, SK_ATTN, s);
  ktrace_start(C, ts, blockIdx.x == 0 && blockIdx.y == 0);
  attn_part<KVT, DH, GP>(C, s, R.slot, (const KVT*)R.ld[s].kv, R.set, blockIdx.y, blockIdx.x);
  ktrace_end(C, ts);
}

// Decode attention of a row block (the PDM's rows: row z at position pos0 + z over the layer's own
// cache). The split is attn_split with the row's scratch. The rows of one (key split, KV head) group
// read the same pages, so they run back to back on one XCD and share its L2: workgroups go to the
// XCDs in turn (workgroup b to XCD b mod 8), and the b-th workgroup of an XCD takes row j mod nrg of
// group (j / nrg) * 8 + xcd, j = b / 8. One-dimensional grid of ceil(groups / 8) * 8 * nrg
// workgroups (groups = max_splits * hkv); the padding groups return at once.
template <typename KVT, int DH, int GP>
__global__ __launch_bounds__(kWG) void k_attn_rows(Ctx C, Rows R, int nrg) {
  extern __shared__ __align__(16) float lds[];
  const int xcd = (int)blockIdx.x & 7, j = (int)blockIdx.x >> 3;
  const int z = j % nrg, grp = (j / nrg) * 8 + xcd;
  if (grp >= C.max_splits * C.hkv) return;
  const int split = grp % C.max_splits, g = grp / C.max_splits;
  const int k0 = split * C.chunk;
  const int page0 = C.page_table[min((k0 + (int)threadIdx.x / kAttnTPK) / C.page, C.max_pages - 1)];
  const Grp gr = resolve(C, R, 0);
  if (!gr.active || z >= gr.nrows) return;
  const int pos0 = gr.pos0 + z;
  const int nsplit = (pos0 + C.chunk) / C.chunk;
  if (split >= nsplit) return;
  const int k1 = min(pos0 + 1, k0 + C.chunk);
  const BufSet& B = C.b[R.set];
  const int cidx = z * C.hkv + g;
  constexpr int RS = kAttnMaxQ * (DH + 2);
  const size_t row = (size_t)(gr.brow0 + z) * C.qdim + g * C.G * DH;
  attn_split_g<KVT, DH, GP>(C, (const KVT*)C.lay[gr.layer].kv, B.q + row, B.ao + row,
                                   B.part + (size_t)cidx * C.max_splits * RS, B.cnt + cidx, g, split, nsplit, k0,
                                   k1, pos0, page0, lds);
}

// Row-block attention on matrix cores (bf16 caches, rows * G <= 32 queries): one workgroup per (key
// split, KV head) serves every row of the block (attn_rows_mfma). Grid: x = key split, y = KV head;
// splits past the block's last key return at once.
template <int DH>
__global__ __launch_bounds__(kWG) void k_attn_rows_mfma(Ctx C, Rows R) {
  extern __shared__ __align__(16) float lds[];
  const Grp gr = resolve(C, R, 0);
  if (!gr.active) return;
  const int split = blockIdx.x, g = blockIdx.y;
  if (split * C.chunk >= gr.pos0 + gr.nrows) return;
  const BufSet& B = C.b[R.set];
  const size_t row0 = (size_t)gr.brow0 * C.qdim;
  attn_rows_mfma<DH>(C, (const uint16_t*)C.lay[gr.layer].kv, B.q + row0, B.ao + row0, B.part, B.cnt, g, split,
                     gr.nrows, gr.pos0, lds);
}

// Launch trace reset.
__global__ __launch_bounds__(kWG) void k_ktrace_reset(Ctx C, int nslots) {
  for (int i = blockIdx.x * kWG + threadIdx.x; i < nslots; i += gridDim.x * kWG) {
    C.ktrace[2 * i] = 0ull;
    C.ktrace[2 * i + 1] = 0ull;
  }
}

// Bandwidth probe: each workgroup streams one contiguous share of the buffer, its threads reading
// consecutive 16-byte blocks with non-temporal loads, eight in flight per thread, folded into one
// value so that no load is dropped.
__global__ __launch_bounds__(kWG) void k_read_probe(const uint4* p, size_t n16, float* sink) {
  constexpr int U = 8;
  const size_t per = (n16 + gridDim.x - 1) / gridDim.x;
  const size_t b0 = (size_t)blockIdx.x * per, b1 = b0 + per < n16 ? b0 + per : n16;
  uint32_t acc = 0;
  for (size_t i0 = b0 + threadIdx.x; i0 < b1; i0 += (size_t)kWG * U) {
    uint4 v[U];
#pragma unroll
    for (int u = 0; u < U; u++) {
      const size_t i = i0 + (size_t)u * kWG;
      v[u] = i < b1 ? ldg16(p + i) : make_uint4(0u, 0u, 0u, 0u);
    }
#pragma unroll
    for (int u = 0; u < U; u++) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  __shared__ uint32_t s_acc;
  if (threadIdx.x == 0) s_acc = 0;
  __syncthreads();
  atomicXor(&s_acc, acc);
  __syncthreads();
  if (threadIdx.x == 0) sink[blockIdx.x] = __uint_as_float(s_acc);
}

void launch_read_probe(const void* buf, size_t n16, float* sink, void* stream) {
  hipLaunchKernelGGL(k_read_probe, dim3(kReadProbeWGs), dim3(kWG), 0, (hipStream_t)stream, (const uint4*)buf, n16, sink);
}

void launch_ktrace_reset(const Ctx& c, int nslots, void* stream) {
  hipLaunchKernelGGL(k_ktrace_reset, dim3((nslots + kWG - 1) / kWG), dim3(kWG), 0, (hipStream_t)stream, c, nslots);
}

// ------------------------------------------------------------------------- embedding / state
template <typename WT>
__device__ __forceinline__ void push_embedding(const Ctx& C, int tok, float* dst0, float* dst1) {
  const WT* E = (const WT*)C.embed + (size_t)tok * C.d;
  for (int k = threadIdx.x; k < C.d; k += kWG) {
    const float v = ld1<WT>(E, k);
    dst0[k] = v;
    if (dst1) dst1[k] = v;
  }
}

template <typename WT>
__global__ __launch_bounds__(kWG) void k_embed_rows(Ctx C, int t0, int nrows) {
  const int i = blockIdx.x;
  if (i >= nrows) return;
  const int tok = C.tok[t0 + i];
  push_embedding<WT>(C, tok, C.pf_x + (size_t)i * C.d, C.pf_anch + (size_t)i * C.n * C.d);
}

// Zero what the next step's kernels count from: both argmax keys. Plain stores: the next launch
// sees them.
__device__ __forceinline__ void reset_step_sync(const Ctx& C) {
  if (threadIdx.x < 2) *C.b[threadIdx.x].hkey = 0ull;
}

// The state update of a step once the target's token y_all (-1 if nothing exits) and the PDM's own
// draft pd_all are known; every thread has read what reset_step_sync clears.
template <typename WT>
__device__ __forceinline__ void verify_update(const Ctx& C, int y_all, int pd_all, int forced_override,
                                              int auto_rb) {
  __shared__ int s_tok, s_pos;
  DevState* st = C.st;
  reset_step_sync(C);
  if (threadIdx.x == 0) {
    const int c = st->c, a = st->a, n = C.n;
    const int pd = pd_all;
    st->pdm_draft = pd;
    st->y = y_all;
    const int dpos = c + a;
    int fd = forced_override;
    if (fd < 0 && dpos < C.max_tokens) fd = C.forced[dpos];
    const int draft = fd >= 0 ? fd : pd;
    spd_step_result r;
    r.decision = SPD_NONE;
    r.target_argmax = -1;
    r.draft = draft;
    r.pdm_draft = pd;
    r.exited_pos = -1;
    r.exited_token = -1;
    r.verified_pos = -1;
    r.verified_token = -1;
    int ptok = -1, ppos = -1;
    if (a == n) {
      const int y = y_all;
      const int succ = n >= 2 ? C.tok[c + 1] : draft;
      r.target_argmax = y;
      r.exited_pos = c;
      r.exited_token = C.tok[c];
      r.verified_pos = c + 1;
      r.verified_token = y;
      st->c = c + 1;
      if (succ == y) {
        r.decision = SPD_ACCEPT;
        C.tok[c + a] = draft;
        ptok = draft;
        ppos = c + a;
      } else {
        r.decision = SPD_REJECT;
        r.draft = -1;
        C.tok[c + 1] = y;
        if (auto_rb) {
          st->a = 1;
          ptok = y;
          ppos = c + 1;
        } else {
          st->a = 0;
          st->pending = 1;
        }
      }
    } else {
      st->a = a + 1;
      C.tok[c + a] = draft;
      ptok = draft;
      ppos = c + a;
    }
    r.committed_len = st->c;
    r.inflight = st->a;
    r.step_index = ++st->nsteps;
    st->res = r;
    C.log[(r.step_index - 1) % kLogCap] = r;
    s_tok = ptok;
    s_pos = ppos;
  }
  __syncthreads();
  if (s_tok >= 0) {
    const int row = s_pos % C.n;
    push_embedding<WT>(C, s_tok, C.resid + (size_t)row * C.d, C.anchors + (size_t)row * C.n * C.d);
  }
}

// Greedy streaming verification (Section 3.4) and the pipeline state update, run by the last
// workgroup of the LM-head launch: the argmax keys were folded in by the launch's other workgroups
// (and by the draft module's own head pass, if it has one), so they are read with device-scope loads.
template <typename WT>
__device__ __forceinline__ void verify_body(const Ctx& C, int forced_override, int auto_rb) {
  DevState* st = C.st;
  const int y_all = (st->a == C.n) ? take_head_dev(C.b[0], C.V) : -1;
  const int pd_all = pdm_token(C, take_head_dev(C.b[1], pdm_rows(C)));
  __syncthreads();  // every thread has read the argmax keys
  verify_update<WT>(C, y_all, pd_all, forced_override, auto_rb);
}


// The fused exit + draft head and verify: every workgroup streams its share of the vocabulary and
// folds its argmax into the keys; once its own key updates have completed it takes a ticket, and the
// workgroup with the last ticket (every other one has finished) runs the verify and resets the
// ticket. Saves the launch of the single-workgroup verify after the head.
// NV 2: the two-row head (src 3); NV 1: the exit row alone (src 0), when the PDM's own pass has left
// its argmax key before this launch.
template <typename WT, int NV>
__global__ __launch_bounds__(kWG) void k_head_verify(Ctx C, int forced_override, int auto_rb) {
  __shared__ int s_last;
  ktrace_start(C, ktrace_extra(C, KT_HEAD), blockIdx.x == 0);
  head_body<WT, NV>(C, NV == 2 ? 3 : 0, 0);
  // the argmax updates are device-scope atomics: once this thread has seen its own complete, the
  // ticket (relaxed, no cache-wide fence) can follow; the last workgroup reads the keys with
  // device-scope loads
  wait_own_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int t = __hip_atomic_fetch_add(&C.st->head_ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (t == (int)gridDim.x - 1);
  }
  __syncthreads();
  ktrace_end(C, ktrace_extra(C, KT_HEAD));
  if (!s_last) return;
  ktrace_start(C, ktrace_extra(C, KT_VERIFY), true);
  verify_body<WT>(C, forced_override, auto_rb);
  if (threadIdx.x == 0) __hip_atomic_store(&C.st->head_ticket, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  ktrace_end(C, ktrace_extra(C, KT_VERIFY));
}

// Sampled decoding (Section 3.4 under sampling, Section 4.1's top-k setting): one workgroup, after
// select_top_k has filled S for the PDM row (and the exit row when a == n). The draft is drawn from
// the PDM's distribution q with the draft position's u_draft (a forced draft has q = delta) and q is
// kept with the token; the exit's distribution p judges the successor: it is kept iff
// u_accept * q(x) < p(x), else the token is drawn from max(0, p - q) (from p if that has no mass)
// with u_resample. Then the ordinary state update runs with that token as the target's. The lookups
// run on wave 0, one distribution entry per lane (k <= 64); the inverse-CDF draws on its lane 0.
template <typename WT>
__device__ __forceinline__ void sampled_verify(const Ctx& C, SelLds& S, int kq, int kp, int forced_override,
                                               int auto_rb) {
  DevState* st = C.st;
  if (threadIdx.x < 64) {
    const int lane = threadIdx.x;
    const int c = st->c, a = st->a, n = C.n;
    const float* u = C.sam.u;
    const int dpos = c + a;
    int fd = forced_override;
    if (fd < 0 && dpos < C.max_tokens) fd = C.forced[dpos];
    int pd = S.ids[1][0];
    if (lane == 0 && dpos < C.max_tokens) pd = S.ids[1][draw_index(S.p[1], kq, u[3 * dpos + 0])];
    pd = __shfl(pd, 0, 64);
    const int draft = fd >= 0 ? fd : pd;
    // the judged token's q: the slot of position c + 1 (n == 1: the distribution just drawn from)
    int qn = 0;
    if (a == n) {
      if (n >= 2) {
        const int r = (c + 1) % n;
        qn = C.sam.q_cnt[r];
        if (lane < qn) {
          S.qj_ids[lane] = C.sam.q_ids[(size_t)r * kMaxTopK + lane];
          S.qj_p[lane] = C.sam.q_p[(size_t)r * kMaxTopK + lane];
        }
      } else if (fd >= 0) {
        qn = 1;
        if (lane == 0) {
          S.qj_ids[0] = fd;
          S.qj_p[0] = 1.0f;
        }
      } else {
        qn = kq;
        if (lane < kq) {
          S.qj_ids[lane] = S.ids[1][lane];
          S.qj_p[lane] = S.p[1][lane];
        }
      }
    }
    {  // keep the new token's q (row dpos mod n; for n >= 2 not the judged row)
      const int r = dpos % n;
      int* qi = C.sam.q_ids + (size_t)r * kMaxTopK;
      float* qp = C.sam.q_p + (size_t)r * kMaxTopK;
      if (fd >= 0) {
        if (lane == 0) {
          qi[0] = fd;
          qp[0] = 1.0f;
          C.sam.q_cnt[r] = 1;
        }
      } else {
        if (lane < kq) {
          qi[lane] = S.ids[1][lane];
          qp[lane] = S.p[1][lane];
        }
        if (lane == 0) C.sam.q_cnt[r] = kq;
      }
    }
    __builtin_amdgcn_wave_barrier();
    int y = -1;
    if (a == n) {
      const int succ = n >= 2 ? C.tok[c + 1] : draft;
      const unsigned long long mp = __ballot(lane < kp && S.ids[0][lane] == succ);
      const unsigned long long mq = __ballot(lane < qn && S.qj_ids[lane] == succ);
      const float px = mp ? S.p[0][__ffsll((long long)mp) - 1] : 0.f;
      const float qx = mq ? S.qj_p[__ffsll((long long)mq) - 1] : 0.f;
      if (u[3 * (c + 1) + 1] * qx < px) {
        y = succ;
      } else {
        float res = 0.f;
        if (lane < kp) {
          const int id = S.ids[0][lane];
          float qv = 0.f;
          for (int j = 0; j < qn; j++)
            if (S.qj_ids[j] == id) qv = S.qj_p[j];
          res = fmaxf(0.f, S.p[0][lane] - qv);
        }
        const float mass = wave_sum(res);
        if (mass > 0.f && lane < kp) S.p[0][lane] = res;
        __builtin_amdgcn_wave_barrier();
        if (lane == 0) y = S.ids[0][draw_index(S.p[0], kp, u[3 * (c + 1) + 2])];
      }
    }
    if (lane == 0) {
      S.out[0] = y;
      S.out[1] = pd;
    }
  }
  __syncthreads();
  const int y = S.out[0], pd = S.out[1];
  __syncthreads();
  verify_update<WT>(C, y, pd, forced_override, auto_rb);
}

// The sampled LM head: head_body with the logits kept, then (last workgroup, as in k_head_verify)
// the top-k selection and the step's sampled verify (NV 2, src 3) or the prefill draw (NV 1, src 2:
// the token at position pos goes to the argmax key of set 0, which the reseed reads).
template <typename WT, int NV>
__global__ __launch_bounds__(kWG) void k_head_sample(Ctx C, int src, int row, int pos, int forced_override,
                                                     int auto_rb, int lcap) {
  extern __shared__ __align__(16) float lds[];
  __shared__ int s_last;
  ktrace_start(C, ktrace_extra(C, KT_HEAD), blockIdx.x == 0);
  head_body<WT, NV, true>(C, src, row, lcap);
  wait_own_stores();
  __syncthreads();
  if (threadIdx.x == 0) {
    const int t = __hip_atomic_fetch_add(&C.st->head_ticket, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (t == (int)gridDim.x - 1);
  }
  __syncthreads();
  ktrace_end(C, ktrace_extra(C, KT_HEAD));
  if (!s_last) return;
  ktrace_start(C, ktrace_extra(C, KT_VERIFY), true);
  SelLds& S = *reinterpret_cast<SelLds*>(lds);  // the staged rows are no longer needed
  if (NV == 2) {
    const int kq = select_top_k(C, 1, S);
    const int kp = C.st->a == C.n ? select_top_k(C, 0, S) : 0;
    sampled_verify<WT>(C, S, kq, kp, forced_override, auto_rb);
  } else if (src == 1) {  // the draft module's own pass: leave q (as target tokens) for the exit row's
    const int kq = select_top_k(C, 1, S);
    for (int j = threadIdx.x; j < kq; j += kWG) {
      const int id = S.ids[1][j];
      __hip_atomic_store(C.sam.pq_ids + j, C.pdm_V > 0 ? C.pdm_map[id] : id, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
      st_dev(C.sam.pq_p + j, S.p[1][j]);
    }
    if (threadIdx.x == 0) __hip_atomic_store(C.sam.pq_cnt, kq, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  } else if (src == 0) {  // the exit row's pass after the draft module's: p, the left q, the verify
    const int kp = C.st->a == C.n ? select_top_k(C, 0, S) : 0;
    const int kq = min(max(ld_dev_i(C.sam.pq_cnt), 1), kMaxTopK);
    for (int j = threadIdx.x; j < kq; j += kWG) {  // (ids kept inside the vocabulary: they are embedded)
      S.ids[1][j] = min(max(ld_dev_i(C.sam.pq_ids + j), 0), C.V - 1);
      S.p[1][j] = ld_dev(C.sam.pq_p + j);
    }
    __syncthreads();
    sampled_verify<WT>(C, S, kq, kp, forced_override, auto_rb);
  } else {
    const int k = select_top_k(C, 0, S);
    if (threadIdx.x == 0) {
      const int x = S.ids[0][draw_index(S.p[0], k, C.sam.u[3 * pos + 2])];
      __hip_atomic_store(C.b[0].hkey, argmax_key(0.0f, x), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
  }
  if (threadIdx.x == 0) __hip_atomic_store(&C.st->head_ticket, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  ktrace_end(C, ktrace_extra(C, KT_VERIFY));
}

// Rollback / first placement: c := keep, one token in flight at position keep (tok < 0: the value
// the last LM-head pass left in st->y).
template <typename WT>
__global__ __launch_bounds__(kWG) void k_reseed(Ctx C, int keep, int tok, int prompt_len) {
  __shared__ int s_tok;
  DevState* st = C.st;
  const int yv = tok >= 0 ? tok : take_head(C.b[0], C.V);
  __syncthreads();  // every thread has read the argmax key
  reset_step_sync(C);
  if (threadIdx.x == 0) {
    const int t = yv;
    if (tok < 0) st->y = t;
    st->c = keep;
    st->a = 1;
    st->pending = 0;
    if (prompt_len >= 0) {
      st->prompt_len = prompt_len;
      st->nsteps = 0;
    }
    C.tok[keep] = t;
    s_tok = t;
  }
  __syncthreads();
  const int row = keep % C.n;
  push_embedding<WT>(C, s_tok, C.resid + (size_t)row * C.d, C.anchors + (size_t)row * C.n * C.d);
}

// -------------------------------------------------------------------------------- launchers
static inline hipStream_t S(void* s) { return (hipStream_t)s; }

// Timing events for the next launches of this host thread (null: plain launches). A timed launch
// hands the events to the dispatch itself, so they hold the kernel's own start and end times.
static thread_local hipEvent_t t_ev_start = nullptr, t_ev_stop = nullptr;
void set_launch_events(void* start, void* stop) {
  t_ev_start = (hipEvent_t)start;
  t_ev_stop = (hipEvent_t)stop;
}
void current_launch_events(hipEvent_t* start, hipEvent_t* stop) {
  *start = t_ev_start;
  *stop = t_ev_stop;
}

template <typename WT>
static inline size_t gemv_lds(int K, int nv) {
  constexpr int BLK = 64 * Elt<WT>::VE;
  const int kp = (K + BLK - 1) / BLK * BLK;
  const int cap = nv == 1 ? kChunkCap1 : kChunkCapN;
  return (size_t)nv * (kp < cap ? kp : cap) * sizeof(float);
}

// Workgroups per stage of a streaming stage launch: about c.stream_wgs (default kStreamWGs) in all, at least enough that no
// wave streams more than 64 pairs (its epilogue values live one per lane), at most one per 4 pairs.
static inline int stream_grid(const Ctx& c, int npairs, int nst) {
  const int total = c.stream_wgs > 0 ? c.stream_wgs : kStreamWGs;
  int wx = (total + nst - 1) / nst;
  wx = std::max(wx, (npairs + 255) / 256);
  wx = std::min(wx, (npairs + 3) / 4);
  return std::max(wx, 1);
}

template <typename WT>
static inline size_t stream_lds(int K) {
  constexpr int BLK = 64 * Elt<WT>::VE;
  return (size_t)(K + BLK - 1) / BLK * BLK * sizeof(float);
}

// Stage launches (r.kind == 0); row blocks go through rows_layer.
template <typename WT>
void Launch<WT>::qkv(const Ctx& c, const Rows& r, void* s) {
  const int np = (c.hq + 2 * c.hkv) * (c.dh / 2);
  launch_timed((k_sgemv<WT, SG_QKV>), dim3(stream_grid(c, np, r.nst), r.nst), dim3(kWG), stream_lds<WT>(c.d), S(s), c, r);
}

template <typename WT>
void Launch<WT>::oproj(const Ctx& c, const Rows& r, void* s) {
  launch_timed((k_sgemv<WT, SG_OPROJ>), dim3(stream_grid(c, (c.d + 1) / 2, r.nst), r.nst), dim3(kWG),
               stream_lds<WT>(c.qdim), S(s), c, r);
}

template <typename WT>
void Launch<WT>::down(const Ctx& c, const Rows& r, void* s) {
  launch_timed((k_sgemv<WT, SG_DOWN>), dim3(stream_grid(c, (c.d + 1) / 2, r.nst), r.nst), dim3(kWG),
               stream_lds<WT>(c.F), S(s), c, r);
}

// Rows of one row-block pass that fit the workgroup's LDS with input width K (at least 1, at most
// max_rows and 8).
struct DevLimits {
  int lds_max = 0, cus = 0;
};
static const DevLimits& dev_limits() {
  static DevLimits L;
  if (L.lds_max == 0) {
    int dev = 0, v = 0, cu = 0;
    if (hipGetDevice(&dev) != hipSuccess ||
        hipDeviceGetAttribute(&v, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) != hipSuccess ||
        hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) {
      v = 65536;
      cu = 256;
    }
    L.lds_max = v;
    L.cus = cu;
  }
  return L;
}

template <typename WT>
static int rows_per_pass(int K, int max_rows) {
  const size_t row = stream_lds<WT>(K);
  const int fit = (int)((size_t)(dev_limits().lds_max - 1024) / row);
  return std::max(1, std::min(std::min(fit, max_rows), kMaxRows));
}

template <typename WT, int KIND>
static void rgemv_launch(const Ctx& c, const Rows& r, int npairs, int K, int max_rows, int cap_wgs, void* s) {
  const int rows = std::max(1, std::min(max_rows, kMaxRows));
  const int min_cols = (npairs + 255) / 256;  // no wave streams more than 64 pairs
  if (cap_wgs <= 0 && stream_lds<WT>(K) * rows > (size_t)kRowLdsBudget && K > kRowSplitK &&
      min_cols <= kRowSplitCols) {
    // K-split (uncapped row blocks: prefill chunks): every chunk of every row in one pass over the
    // weights, a small LDS slice per workgroup. A capped launch (side work beside the stage compute)
    // keeps the full-width form: with few columns the split's last-arriver merges run long.
    const int ns = (K + kRowSplitK - 1) / kRowSplitK;
    const size_t shm = (size_t)rows * kRowSplitK * sizeof(float);
    const int resident = dev_limits().cus * std::max(1, (int)((size_t)dev_limits().lds_max / (shm + 1024)));
    const int cols = std::min(std::max(std::min(stream_grid(c, npairs, 1), std::max(1, resident / ns)), min_cols),
                              kRowSplitCols);
    const dim3 grid(cols, ns);
    if (rows <= 4)
      launch_timed((k_rgemv_ks<WT, KIND, 4>), grid, dim3(kWG), shm, S(s), c, r);
    else
      launch_timed((k_rgemv_ks<WT, KIND, 8>), grid, dim3(kWG), shm, S(s), c, r);
    return;
  }
  const int nrp = rows_per_pass<WT>(K, max_rows);
  const size_t shm = stream_lds<WT>(K) * nrp;
  // no more workgroups than the GPU holds at once with this much LDS (a second round would double
  // the launch), and enough waves that none streams more than 64 pairs
  const int resident = dev_limits().cus * std::max(1, (int)((size_t)dev_limits().lds_max / (shm + 1024)));
  int wgs = std::min(stream_grid(c, npairs, 1), resident);
  if (cap_wgs > 0) wgs = std::min(wgs, cap_wgs);  // side work: leave most CUs to the stages
  wgs = std::max(wgs, (npairs + 255) / 256);
  const dim3 grid(wgs);
  if (nrp <= 4)
    launch_timed((k_rgemv<WT, KIND, 4>), grid, dim3(kWG), shm, S(s), c, r, nrp);
  else
    launch_timed((k_rgemv<WT, KIND, 8>), grid, dim3(kWG), shm, S(s), c, r, nrp);
}

template <typename WT>
void Launch<WT>::rows_layer(const Ctx& c, const Rows& r, int max_rows, int cap_wgs, void* s) {
  for (int k = 0; k < 5; k++) rows_sublayer(c, r, max_rows, k, cap_wgs, s);
}

template <typename WT>
void Launch<WT>::rows_sublayer(const Ctx& c, const Rows& r, int max_rows, int k, int cap_wgs, void* s) {
  max_rows = std::max(1, std::min(max_rows, kMaxRows));
  if (k == 0) rgemv_launch<WT, SG_QKV>(c, r, (c.hq + 2 * c.hkv) * (c.dh / 2), c.d, max_rows, cap_wgs, s);
  if (k == 2) rgemv_launch<WT, SG_OPROJ>(c, r, (c.d + 1) / 2, c.qdim, max_rows, cap_wgs, s);
  if (k == 3) rgemv_launch<WT, SG_GATEUP>(c, r, c.F, c.d, max_rows, cap_wgs, s);
  if (k == 4) rgemv_launch<WT, SG_DOWN>(c, r, (c.d + 1) / 2, c.F, max_rows, cap_wgs, s);
  if (k != 1) return;
  if constexpr (std::is_same<WT, uint16_t>::value) {
    if (max_rows * c.G <= 32 && (c.dh == 64 || c.dh == 128)) {  // every query of the block in one MFMA tile
      const dim3 grid(c.max_splits, c.hkv);
      if (c.dh == 128)
        launch_timed((k_attn_rows_mfma<128>), grid, dim3(kWG), attn_rows_mfma_lds<128>(), S(s), c, r);
      else
        launch_timed((k_attn_rows_mfma<64>), grid, dim3(kWG), attn_rows_mfma_lds<64>(), S(s), c, r);
      return;
    }
  }
  const int groups8 = (c.max_splits * c.hkv + 7) / 8 * 8;  // see k_attn_rows: XCD-aware order
  const dim3 agrid(groups8 * max_rows);
  const bool g4 = c.G <= 4;
  if (c.dh == 128) {
    if (g4)
      launch_timed((k_attn_rows<WT, 128, 4>), agrid, dim3(kWG), attn_split_lds<WT, 128>(), S(s), c, r, max_rows);
    else
      launch_timed((k_attn_rows<WT, 128, 8>), agrid, dim3(kWG), attn_split_lds<WT, 128>(), S(s), c, r, max_rows);
  } else {
    if (g4)
      launch_timed((k_attn_rows<WT, 64, 4>), agrid, dim3(kWG), attn_split_lds<WT, 64>(), S(s), c, r, max_rows);
    else
      launch_timed((k_attn_rows<WT, 64, 8>), agrid, dim3(kWG), attn_split_lds<WT, 64>(), S(s), c, r, max_rows);
  }
}

template <typename WT>
void Launch<WT>::gateup(const Ctx& c, const Rows& r, void* s) {
  launch_timed((k_sgemv<WT, SG_GATEUP>), dim3(stream_grid(c, c.F, r.nst), r.nst), dim3(kWG), stream_lds<WT>(c.d),
               S(s), c, r);
}

template <typename WT>
void Launch<WT>::attn(const Ctx& c, const Rows& r, void* s) {
  const dim3 grid(c.max_splits, c.hkv, r.nst);
  const bool g4 = c.G <= 4;
  if (c.dh == 128) {
    if (g4)
      launch_timed((k_attn_stage<WT, 128, 4>), grid, dim3(kWG), attn_split_lds<WT, 128>(), S(s), c, r);
    else
      launch_timed((k_attn_stage<WT, 128, 8>), grid, dim3(kWG), attn_split_lds<WT, 128>(), S(s), c, r);
  } else {
    if (g4)
      launch_timed((k_attn_stage<WT, 64, 4>), grid, dim3(kWG), attn_split_lds<WT, 64>(), S(s), c, r);
    else
      launch_timed((k_attn_stage<WT, 64, 8>), grid, dim3(kWG), attn_split_lds<WT, 64>(), S(s), c, r);
  }
}

template <typename WT>
void Launch<WT>::pdm_fc(const Ctx& c, int prefill, int nrows, void* s) {
  const dim3 grid((c.d + 7) / 8);
  launch_timed((k_pdm_fc<WT>), grid, dim3(kWG), gemv_lds<WT>(c.n * c.d, kMaxRows), S(s), c, prefill, nrows);
}

// Workgroups of `fn` (with `lds` bytes of dynamic LDS) that the GPU holds at once.
static int resident_wgs(const void* fn, size_t lds) {
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, kWG, lds) != hipSuccess || per_cu < 1) per_cu = 1;
  return per_cu * dev_limits().cus;
}

template <typename WT>
void Launch<WT>::head(const Ctx& c, int src, int row, void* s) {
  // a wave streams its vocabulary pairs back to back; no more workgroups than the GPU holds at once,
  // since the head runs alone and a second round of workgroups would only add a tail
  constexpr int BLK = 64 * Elt<WT>::VE;
  const size_t kl_pad = (size_t)(c.d + BLK - 1) / BLK * BLK;
  const int np = ((src == 1 && c.pdm_V > 0 ? c.pdm_V : c.V) + 1) / 2;
  if (src == 3) {
    const size_t shm = 2 * kl_pad * sizeof(float);
    const int res = resident_wgs((const void*)k_head<WT, 2>, shm);
    const dim3 grid(std::max(std::min(stream_grid(c, np, 1), res), 1));
    launch_timed((k_head<WT, 2>), grid, dim3(kWG), shm, S(s), c, src, row);
  } else {
    const size_t shm = kl_pad * sizeof(float);
    const int res = resident_wgs((const void*)k_head<WT, 1>, shm);
    const dim3 grid(std::max(std::min(stream_grid(c, np, 1), res), 1));
    launch_timed((k_head<WT, 1>), grid, dim3(kWG), shm, S(s), c, src, row);
  }
}

template <typename WT>
void Launch<WT>::head_verify(const Ctx& c, int two_rows, int forced_override, int auto_rb, void* s) {
  constexpr int BLK = 64 * Elt<WT>::VE;
  const int nv = two_rows ? 2 : 1;
  const size_t shm = nv * (size_t)(c.d + BLK - 1) / BLK * BLK * sizeof(float);
  const void* fn = two_rows ? (const void*)k_head_verify<WT, 2> : (const void*)k_head_verify<WT, 1>;
  const int res = resident_wgs(fn, shm);
  const dim3 grid(std::max(std::min(stream_grid(c, (c.V + 1) / 2, 1), res), 1));
  if (two_rows)
    launch_timed((k_head_verify<WT, 2>), grid, dim3(kWG), shm, S(s), c, forced_override, auto_rb);
  else
    launch_timed((k_head_verify<WT, 1>), grid, dim3(kWG), shm, S(s), c, forced_override, auto_rb);
}

template <typename WT>
void Launch<WT>::head_sample(const Ctx& c, int src, int row, int pos, int forced_override, int auto_rb, void* s) {
  // dynamic LDS: the staged rows and the waves' logit regions during the pass, the selection's state
  // afterwards; a smaller grid (fewer resident workgroups) means larger regions, so settle both
  constexpr int BLK = 64 * Elt<WT>::VE;
  const size_t kl_pad = (size_t)(c.d + BLK - 1) / BLK * BLK;
  const int np = ((src == 1 && c.pdm_V > 0 ? c.pdm_V : c.V) + 1) / 2;
  const int nv = src == 3 ? 2 : 1;
  const void* fn = src == 3 ? (const void*)k_head_sample<WT, 2> : (const void*)k_head_sample<WT, 1>;
  int grid = std::max(std::min(stream_grid(c, np, 1), kSampleWGs), 1);
  int lcap = 0;
  size_t shm = 0;
  for (int it = 0; it < 4; it++) {
    lcap = 2 * ((np + 4 * grid - 1) / (4 * grid));
    shm = std::max(((size_t)nv * kl_pad + (size_t)nv * 4 * lcap) * sizeof(float), sizeof(SelLds));
    const int res = resident_wgs(fn, shm);
    if (res >= grid) break;
    grid = std::max(res, 1);
  }
  // lcap is the region each launch's wave needs; the kernel stores directly if its region exceeds it
  if (src == 3)
    launch_timed((k_head_sample<WT, 2>), dim3(grid), dim3(kWG), shm, S(s), c, src, row, pos, forced_override,
                 auto_rb, lcap);
  else
    launch_timed((k_head_sample<WT, 1>), dim3(grid), dim3(kWG), shm, S(s), c, src, row, pos, forced_override,
                 auto_rb, lcap);
}

template <typename WT>
void Launch<WT>::embed_rows(const Ctx& c, int t0, int nrows, void* s) {
  launch_timed((k_embed_rows<WT>), dim3(nrows), dim3(kWG), 0, S(s), c, t0, nrows);
}

template struct Launch<float>;
template struct Launch<uint16_t>;

void launch_reseed(const Ctx& c, int keep, int tok, int prompt_len, void* s, int bf16) {
  if (bf16)
    launch_timed((k_reseed<uint16_t>), dim3(1), dim3(kWG), 0, S(s), c, keep, tok, prompt_len);
  else
    launch_timed((k_reseed<float>), dim3(1), dim3(kWG), 0, S(s), c, keep, tok, prompt_len);
}

}  // namespace spd
