// Sampled decoding on the device: exact top-k selection over the logits a sampled LM-head launch
// leaves behind, the top-k temperature softmax, inverse-CDF draws and the rejection-sampling
// verify (Section 3.4 under sampling; Section 4.1 fixes T = 1, top-k 50, top-p 1.0).
//
// Selection runs in the last workgroup of the launch. Keys are the 64-bit argmax keys (logit
// descending, then index ascending), so every key is distinct and "the k largest keys" is exactly
// the top-k with ties broken towards the lower index. Each workgroup of the head left its best key
// per row; the k-th largest of those maxima, t_lo, is a lower bound of the k-th largest logit key
// overall (k workgroups each hold a key >= t_lo). Only workgroups whose maximum reaches t_lo can
// hold a top-k key, and only their entries >= t_lo are candidates: typically little more than k.
// A radix select (8-bit digits, most significant first) finds the k-th largest candidate key T, and
// the k keys >= T are sorted by rank.
#pragma once
#include "spd_dev.h"
#include "spd_devfn.h"

namespace spd {

struct SelLds {
  unsigned long long keys[kSelCap];  // workgroup maxima, then candidates
  unsigned long long top[kMaxTopK];
  int sel[kSampleWGs];               // workgroups whose maximum reaches t_lo
  unsigned hist[256];
  int misc[4];
  int ids[2][kMaxTopK];              // [0]: target row, [1]: PDM row (value-descending order)
  float p[2][kMaxTopK];
  int out[2];
};

__device__ __forceinline__ unsigned long long ld_dev_u64(const unsigned long long* p) {
  return __hip_atomic_load(const_cast<unsigned long long*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// The logit a key was made from (inverse of argmax_key's monotone map).
__device__ __forceinline__ float key_value(unsigned long long key) {
  uint32_t u = (uint32_t)(key >> 32);
  u = (u & 0x80000000u) ? (u & 0x7fffffffu) : ~u;
  return __uint_as_float(u);
}

// The k-th largest of the keys that visit(f) hands to f (each thread calls f for its share);
// requires 1 <= k <= number of keys. Whole workgroup; uses S.hist and S.misc[0..1].
template <typename Visit>
__device__ unsigned long long select_kth(Visit visit, int k, SelLds& S) {
  const int tid = threadIdx.x, lane = tid & 63;
  unsigned long long prefix = 0ull, mask = 0ull;
  for (int shift = 56; shift >= 0; shift -= 8) {
    S.hist[tid] = 0u;  // kWG == 256 bins
    __syncthreads();
    visit([&](unsigned long long key) {
      if ((key & mask) == prefix) atomicAdd(&S.hist[(key >> shift) & 255u], 1u);
    });
    __syncthreads();
    if (tid < 64) {
      // lane l holds bins 4l..4l+3; suf = keys in bins >= 4l
      const unsigned b0 = S.hist[4 * lane], b1 = S.hist[4 * lane + 1], b2 = S.hist[4 * lane + 2],
                     b3 = S.hist[4 * lane + 3];
      const unsigned own = b0 + b1 + b2 + b3;
      unsigned suf = own;
#pragma unroll
      for (int off = 1; off < 64; off <<= 1) {
        const unsigned t = __shfl_down(suf, off);
        if (lane + off < 64) suf += t;
      }
      const unsigned above = suf - own, kk = (unsigned)k;
      if (above < kk && kk <= suf) {
        unsigned acc = above;
        int dig;
        if (acc + b3 >= kk) {
          dig = 4 * lane + 3;
        } else if ((acc += b3) + b2 >= kk) {
          dig = 4 * lane + 2;
        } else if ((acc += b2) + b1 >= kk) {
          dig = 4 * lane + 1;
        } else {
          acc += b1;
          dig = 4 * lane;
        }
        S.misc[0] = dig;
        S.misc[1] = (int)acc;  // keys in the digits above
      }
    }
    __syncthreads();
    prefix |= (unsigned long long)S.misc[0] << shift;
    mask |= 0xffull << shift;
    k -= S.misc[1];
    __syncthreads();
  }
  return prefix;
}

// Every logit key of row `set` in the regions of the workgroups listed in S.sel[0..nsel) that is
// >= tlo, handed to f (each thread its share). The region geometry is the head's (see Sampler).
template <typename F>
__device__ void visit_regions(const Ctx& C, int set, const SelLds& S, int nsel, unsigned long long tlo, F f) {
  const int V = C.V, NW = (int)gridDim.x * 4, npairs = (V + 1) / 2;
  const int cmax = 2 * ((npairs + NW - 1) / NW);
  const int per = 4 * cmax;
  const int total = nsel * per;
  const float* base = C.sam.wlog + (size_t)set * C.sam.wlog_stride;
  for (int e = threadIdx.x; e < total; e += kWG) {
    const int off = e % per;
    const int wv = S.sel[e / per] * 4 + off / cmax, i = off % cmax;
    const int cnt = wv < npairs ? (npairs - 1 - wv) / NW + 1 : 0;
    const int m = 2 * (wv + (i >> 1) * NW) + (i & 1);
    if (i >= 2 * cnt || m >= V) continue;
    const unsigned long long key = argmax_key(ld_dev(base + (size_t)wv * cmax + i), m);
    if (key >= tlo) f(key);
  }
}

// Top-k distribution of row `set` (0 target, 1 PDM) into S.ids[set] / S.p[set]: the k = min(top_k,
// V) largest logits, value descending (lower index first among equal values), and their softmax at
// temperature 1/inv_temp (max-subtracted, fp32). Whole workgroup; returns k.
__device__ int select_top_k(const Ctx& C, int set, SelLds& S) {
  const int tid = threadIdx.x, G = (int)gridDim.x, V = C.V;
  const int k = min(C.sam.top_k, V);
  for (int i = tid; i < G; i += kWG) S.keys[i] = ld_dev_u64(C.sam.wgmax + (size_t)set * kSampleWGs + i);
  __syncthreads();
  unsigned long long tlo = 1ull;  // every real key is >= 1
  if (G >= k) {
    const unsigned long long t = select_kth([&](auto f) { for (int i = tid; i < G; i += kWG) f(S.keys[i]); }, k, S);
    tlo = t > 1ull ? t : 1ull;
  }
  if (tid == 0) {
    S.misc[2] = 0;
    S.misc[3] = 0;
  }
  __syncthreads();
  for (int i = tid; i < G; i += kWG)
    if (S.keys[i] >= tlo) S.sel[atomicAdd(&S.misc[2], 1)] = i;
  __syncthreads();
  const int nsel = S.misc[2];
  visit_regions(C, set, S, nsel, tlo, [&](unsigned long long key) {
    const int at = atomicAdd(&S.misc[3], 1);
    if (at < kSelCap) S.keys[at] = key;
  });
  __syncthreads();
  const int ncand = S.misc[3];
  const bool in_lds = ncand <= kSelCap;
  auto cands = [&](auto f) {
    if (in_lds) {
      for (int i = tid; i < ncand; i += kWG) f(S.keys[i]);
    } else {
      visit_regions(C, set, S, nsel, tlo, f);
    }
  };
  const unsigned long long T = select_kth(cands, k, S);
  if (tid == 0) S.misc[2] = 0;
  __syncthreads();
  cands([&](unsigned long long key) {
    if (key >= T) {
      const int at = atomicAdd(&S.misc[2], 1);
      if (at < kMaxTopK) S.top[at] = key;
    }
  });
  __syncthreads();
  // exactly k distinct keys are >= T; each one's rank is its place in value-descending order
  unsigned long long mine = 0ull;
  int rank = 0;
  if (tid < k) {
    mine = S.top[tid];
    for (int j = 0; j < k; j++) rank += S.top[j] > mine;
    S.ids[set][rank] = argmax_index(mine, V);
    S.p[set][rank] = key_value(mine);
  }
  __syncthreads();
  const float top = S.p[set][0];
  const float w = tid < k ? expf((S.p[set][tid] - top) * C.sam.inv_temp) : 0.f;
  __syncthreads();
  if (tid < k) S.p[set][tid] = w;
  __syncthreads();
  if (tid == 0) {
    float sum = 0.f;
    for (int j = 0; j < k; j++) sum += S.p[set][j];
    const float inv = 1.0f / sum;
    for (int j = 0; j < k; j++) S.p[set][j] *= inv;
  }
  __syncthreads();
  return k;
}

// Inverse CDF over nonnegative weights w[0..m) in their order: the first i with u*sum < cumsum_i
// (the last entry if rounding leaves none). One thread.
__device__ __forceinline__ int draw_index(const float* w, int m, float u) {
  float sum = 0.f;
  for (int i = 0; i < m; i++) sum += w[i];
  const float t = u * sum;
  float cs = 0.f;
  for (int i = 0; i < m; i++) {
    cs += w[i];
    if (t < cs) return i;
  }
  return m - 1;
}

__device__ __forceinline__ float prob_in(const int* ids, const float* p, int m, int tok) {
  for (int j = 0; j < m; j++)
    if (ids[j] == tok) return p[j];
  return 0.f;
}

}  // namespace spd
