// Decode attention of one stage's token over one KV head's paged cache, one key split per workgroup
// (the stage launches, the mixed launches and the persistent step kernel share it, so all compute the
// same bits).
//
// The token at position pos0 attends to keys 0..pos0 of its own layer (Section 3.1: each stage's
// token reads the cache of the layer it is on). Its G query heads share KV head g (grouped-query
// attention). A split covers keys [k0, k1) in passes of 64 keys: thread t owns key t/4 of a pass and
// a quarter of its head dimension, for K (registers) and V (LDS tile) alike, so one page-table lookup
// serves both, and the next pass's keys are requested before the current pass is computed. Softmax
// is online across passes; the split ends with its (o, m, l). With one split the workgroup writes the
// output; otherwise the split that finishes last (a ticket per stage and head) merges every split in
// split order: all (m, l) pairs are read at once, the split weights exp(m - M) / L go to LDS, and the
// partial outputs are summed in split order with their loads issued eight at a time. The split size is
// a function of the configuration only, so a token's result never depends on how many stages run.
#pragma once
#include "spd_devfn.h"

namespace spd {

constexpr int kAttnTPK = 4;                // threads per key
constexpr int kAttnPass = kWG / kAttnTPK;  // keys per pass
constexpr int kAttnMaxQ = 8;               // query heads per KV head

template <typename KVT, int DH>
constexpr size_t attn_split_lds() {
  return (size_t)kAttnMaxQ * DH * 4 + (size_t)kAttnMaxQ * kAttnPass * 4 + (size_t)kAttnPass * DH * sizeof(KVT) +
         (size_t)2 * kMaxSplits * kAttnMaxQ * 4;
}

// 16 bytes (16-byte aligned) with device-scope loads.
__device__ __forceinline__ uint4 ldg16_coherent(const void* p) {
  unsigned long long* q = (unsigned long long*)const_cast<void*>(p);
  const unsigned long long a = __hip_atomic_load(q, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  const unsigned long long b = __hip_atomic_load(q + 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_uint4((uint32_t)a, (uint32_t)(a >> 32), (uint32_t)b, (uint32_t)(b >> 32));
}

// KV cache reads. Ordinary loads: a pass's keys come back faster than with the non-temporal hint.
__device__ __forceinline__ uint4 ldkv16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ void st_dev2f(float* p, float x, float y) {  // p 8-byte aligned
  const unsigned long long u = (unsigned long long)__float_as_uint(x) | ((unsigned long long)__float_as_uint(y) << 32);
  __hip_atomic_store((unsigned long long*)p, u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// One split. COH: the query and the newest key (pos0) were written by the same launch (device-scope
// loads) and the output goes to a tile of the same launch (device-scope stores). kv: the layer's
// cache; q: the G rotated query rows of this head group; out: their G output rows; rec: the
// (o[8][DH], m[8], l[8]) records of this (stage, head), one per split; cnt: its split ticket (zero at
// rest); page0: the physical page of this thread's key in the first pass (requested by the caller
// before anything else). Returns true when this workgroup wrote the final output.
template <typename KVT, int DH, bool COH>
__device__ bool attn_split(const Ctx& C, const KVT* kvb, const float* q, float* out, float* rec_base, int* cnt, int g,
                           int split, int nsplit, int k0, int k1, int pos0, int page0, float* lds) {
  constexpr int TPK = kAttnTPK, NE = DH / TPK, VE = Elt<KVT>::VE, KCH = NE / VE;
  constexpr int MAXQ = kAttnMaxQ, PASS = kAttnPass;
  constexpr int RS = MAXQ * (DH + 2);
  float* qs = lds;                                         // [MAXQ][DH] pre-scaled queries
  float* sc = qs + MAXQ * DH;                              // [MAXQ][PASS] scores, then probabilities
  KVT* vs = reinterpret_cast<KVT*>(sc + MAXQ * PASS);      // [PASS][DH] V tile
  float* s_pw = reinterpret_cast<float*>(vs + PASS * DH);  // merge: m of each split, then its weight
  float* s_pl = s_pw + kMaxSplits * MAXQ;
  __shared__ float s_m[MAXQ], s_l[MAXQ], s_al[MAXQ];
  __shared__ int s_last;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int kk = tid / TPK, qq = tid % TPK;
  const int G = C.G;
  const size_t page_elems = (size_t)2 * C.hkv * C.page * DH;
  const size_t head_off = (size_t)g * C.page * DH;
  const size_t voff = (size_t)C.hkv * C.page * DH;
  uint4 kraw[KCH], vraw[KCH];
  auto issue = [&](int kp, int page) {
    const int key = kp + kk;
    if (key < k1) {
      const KVT* base = kvb + (size_t)page * page_elems + head_off + (size_t)(key % C.page) * DH + qq * NE;
      if (COH && key == pos0) {
#pragma unroll
        for (int c4 = 0; c4 < KCH; c4++) kraw[c4] = ldg16_coherent(reinterpret_cast<const uint4*>(base) + c4);
#pragma unroll
        for (int c4 = 0; c4 < KCH; c4++) vraw[c4] = ldg16_coherent(reinterpret_cast<const uint4*>(base + voff) + c4);
      } else {
#pragma unroll
        for (int c4 = 0; c4 < KCH; c4++) kraw[c4] = ldkv16(reinterpret_cast<const uint4*>(base) + c4);
#pragma unroll
        for (int c4 = 0; c4 < KCH; c4++) vraw[c4] = ldkv16(reinterpret_cast<const uint4*>(base + voff) + c4);
      }
    }
  };
  issue(k0, page0);
  for (int e = tid; e < G * DH; e += kWG) qs[e] = (COH ? ld_dev(q + e) : q[e]) * C.scale;
  if (tid < MAXQ) {
    s_m[tid] = -INFINITY;
    s_l[tid] = 0.f;
  }
  constexpr int npair = DH >> 1;
  constexpr int NG = kWG / npair;
  constexpr int MAXU = (MAXQ + NG - 1) / NG;
  const int dp = tid % npair, qg = tid / npair;
  float o0[MAXU], o1[MAXU];
#pragma unroll
  for (int u = 0; u < MAXU; u++) o0[u] = o1[u] = 0.f;
  for (int kp = k0; kp < k1; kp += PASS) {
    const int nk = min(PASS, k1 - kp);
    float kr[NE];
    if (kk < nk) {
#pragma unroll
      for (int c4 = 0; c4 < KCH; c4++) reinterpret_cast<uint4*>(vs + kk * DH + qq * NE)[c4] = vraw[c4];
#pragma unroll
      for (int c4 = 0; c4 < KCH; c4++) unpack16<KVT>(kraw[c4], kr + c4 * VE);
    }
    if (kp + PASS < k1) {  // the next pass's keys are in flight while this one is computed
      const int nkey = kp + PASS + kk;
      issue(kp + PASS, C.page_table[min(nkey, k1 - 1) / C.page]);
    }
    __syncthreads();  // q staged (first pass), V tile written
    for (int qi = 0; qi < G; qi++) {
      float dsum = 0.f;
      if (kk < nk) {
        const float* qv = qs + qi * DH + qq * NE;
#pragma unroll
        for (int e = 0; e < NE; e += 4) {
          const float4 q4 = *reinterpret_cast<const float4*>(qv + e);
          dsum = fmaf(q4.x, kr[e], dsum);
          dsum = fmaf(q4.y, kr[e + 1], dsum);
          dsum = fmaf(q4.z, kr[e + 2], dsum);
          dsum = fmaf(q4.w, kr[e + 3], dsum);
        }
      }
      dsum += __shfl_xor(dsum, 1, 64);
      dsum += __shfl_xor(dsum, 2, 64);
      if (qq == 0 && kk < nk) sc[qi * PASS + kk] = dsum;
    }
    __syncthreads();
    for (int qi = w; qi < G; qi += kWG / 64) {  // online softmax, one wave per query head
      const float sv = lane < nk ? sc[qi * PASS + lane] : -INFINITY;
      const float mx = wave_max(sv);
      const float mo = s_m[qi];
      const float mn = fmaxf(mo, mx);
      const float p = lane < nk ? expf(sv - mn) : 0.f;
      if (lane < nk) sc[qi * PASS + lane] = p;
      const float ps = wave_sum(p);
      if (lane == 0) {
        const float al = (mo == -INFINITY) ? 0.f : expf(mo - mn);
        s_al[qi] = al;
        s_l[qi] = s_l[qi] * al + ps;
        s_m[qi] = mn;
      }
    }
    __syncthreads();
#pragma unroll
    for (int u = 0; u < MAXU; u++) {
      const int qi = qg + u * NG;
      if (qi < G) {
        const float al = s_al[qi];
        o0[u] *= al;
        o1[u] *= al;
      }
    }
    // P.V: eight keys' V pairs and probabilities are read from LDS together (rows >= nk of the
    // tile hold stale values and are skipped), then accumulated in key order
    for (int k2 = 0; k2 < nk; k2 += 8) {
      float2 vv[8];
#pragma unroll
      for (int j = 0; j < 8; j++) vv[j] = ld2<KVT>(vs + (size_t)(k2 + j) * DH + 2 * dp);
#pragma unroll
      for (int u = 0; u < MAXU; u++) {
        const int qi = qg + u * NG;
        if (qi < G) {
          float pp[8];
#pragma unroll
          for (int j = 0; j < 8; j++) pp[j] = sc[qi * PASS + k2 + j];
#pragma unroll
          for (int j = 0; j < 8; j++) {
            if (k2 + j < nk) {
              o0[u] = fmaf(pp[j], vv[j].x, o0[u]);
              o1[u] = fmaf(pp[j], vv[j].y, o1[u]);
            }
          }
        }
      }
    }
    __syncthreads();
  }
  if (nsplit == 1) {
#pragma unroll
    for (int u = 0; u < MAXU; u++) {
      const int qi = qg + u * NG;
      if (qi < G) {
        const float inv = 1.0f / s_l[qi];
        if (COH) {
          st_dev2f(out + qi * DH + 2 * dp, o0[u] * inv, o1[u] * inv);
        } else {
          out[qi * DH + 2 * dp] = o0[u] * inv;
          out[qi * DH + 2 * dp + 1] = o1[u] * inv;
        }
      }
    }
    return true;
  }
  float* rec = rec_base + (size_t)split * RS;
#pragma unroll
  for (int u = 0; u < MAXU; u++) {
    const int qi = qg + u * NG;
    if (qi < G) {
      st_dev(rec + qi * DH + 2 * dp, o0[u]);
      st_dev(rec + qi * DH + 2 * dp + 1, o1[u]);
    }
  }
  if (tid < G) {
    st_dev(rec + MAXQ * DH + tid, s_m[tid]);
    st_dev(rec + MAXQ * DH + MAXQ + tid, s_l[tid]);
  }
  wait_own_stores();
  __syncthreads();
  if (tid == 0) {
    const int t = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (t == nsplit - 1);
  }
  __syncthreads();
  if (!s_last) return false;
  for (int e = tid; e < nsplit * G; e += kWG) {  // every split has >= 1 key, so m is finite
    const int sp = e / G, qi = e % G;
    s_pw[sp * MAXQ + qi] = ld_dev(rec_base + (size_t)sp * RS + MAXQ * DH + qi);
    s_pl[sp * MAXQ + qi] = ld_dev(rec_base + (size_t)sp * RS + MAXQ * DH + MAXQ + qi);
  }
  __syncthreads();
  if (tid < G) {  // split order, fixed
    float M = -INFINITY;
    for (int sp = 0; sp < nsplit; sp++) M = fmaxf(M, s_pw[sp * MAXQ + tid]);
    float Ls = 0.f;
    for (int sp = 0; sp < nsplit; sp++) Ls = fmaf(s_pl[sp * MAXQ + tid], expf(s_pw[sp * MAXQ + tid] - M), Ls);
    s_m[tid] = M;
    s_l[tid] = 1.0f / Ls;
  }
  __syncthreads();
  for (int e = tid; e < nsplit * G; e += kWG) {
    const int sp = e / G, qi = e % G;
    s_pw[sp * MAXQ + qi] = expf(s_pw[sp * MAXQ + qi] - s_m[qi]) * s_l[qi];
  }
  __syncthreads();
#pragma unroll
  for (int u = 0; u < MAXU; u++) {
    const int qi = qg + u * NG;
    if (qi < G) {
      float A0 = 0.f, A1 = 0.f;
      for (int sp0 = 0; sp0 < nsplit; sp0 += 8) {
        float2 v[8];
#pragma unroll
        for (int j = 0; j < 8; j++)
          v[j] = sp0 + j < nsplit ? ld_dev2(rec_base + (size_t)(sp0 + j) * RS + qi * DH + 2 * dp) : make_float2(0.f, 0.f);
#pragma unroll
        for (int j = 0; j < 8; j++) {
          if (sp0 + j < nsplit) {
            const float f = s_pw[(sp0 + j) * MAXQ + qi];
            A0 = fmaf(v[j].x, f, A0);
            A1 = fmaf(v[j].y, f, A1);
          }
        }
      }
      if (COH) {
        st_dev2f(out + qi * DH + 2 * dp, A0, A1);
      } else {
        out[qi * DH + 2 * dp] = A0;
        out[qi * DH + 2 * dp + 1] = A1;
      }
    }
  }
  if (tid == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

}  // namespace spd
