// Sampled decoding on the device: exact top-k selection over the logits a sampled LM-head launch
// leaves behind, the top-k temperature softmax, inverse-CDF draws and the rejection-sampling
// verify (Section 3.4 under sampling; Section 4.1 fixes T = 1, top-k 50, top-p 1.0).
//
// Selection runs in the last workgroup of the launch. Keys are the 64-bit argmax keys (logit
// descending, then index ascending), so every key is distinct and "the k largest keys" is exactly
// the top-k with ties broken towards the lower index. Each workgroup of the head left its best key
// per row; each thread takes the largest of up to four of those maxima, and the k-th largest of the
// threads' values, t_lo, is a lower bound of the k-th largest logit key overall (k threads each saw
// a distinct key >= t_lo). Only workgroups whose maximum reaches t_lo can hold a top-k key, and only
// their entries >= t_lo are candidates: typically little more than k. Each candidate's rank is the
// number of candidates above it, so the top-k land in rank order with no further passes. (Over
// kSelCap candidates a radix select over memory, 8-bit digits most significant first, finds the
// k-th largest key instead.)
#pragma once
#include "spd_dev.h"
#include "spd_devfn.h"

namespace spd {

static_assert(kSampleWGs % kWG == 0 && kSampleWGs / kWG <= 4, "workgroup maxima per selection thread");

struct SelLds {
  unsigned long long keys[kSelCap];  // workgroup maxima, then candidates
  unsigned long long top[kMaxTopK];
  unsigned long long gmax[kWG];      // each thread's largest workgroup maximum
  int sel[kSampleWGs];               // workgroups whose maximum reaches t_lo
  unsigned hist[256];
  int misc[4];
  unsigned long long tlo;
  int ids[2][kMaxTopK];              // [0]: target row, [1]: PDM row (value-descending order)
  float p[2][kMaxTopK];
  int qj_ids[kMaxTopK];              // the draft distribution of the token being judged
  float qj_p[kMaxTopK];
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

// Vocabulary rows of a set's head: the draft module's own head for set 1 when it has one.
__device__ __forceinline__ int set_rows(const Ctx& C, int set) {
  return set == 1 && C.pdm_V > 0 ? C.pdm_V : C.V;
}

// Every logit key of row `set` in the regions of the workgroups listed in S.sel[0..nsel) that is
// >= tlo, handed to f (each thread its share). The region geometry is the head's (see Sampler): a
// workgroup's four wave regions are consecutive, 4 * cmax floats (cmax even), so the entries go as
// 8-byte pairs, eight device-scope loads in flight per thread before any is looked at.
template <typename F>
__device__ void visit_regions(const Ctx& C, int set, const SelLds& S, int nsel, unsigned long long tlo, F f) {
  const int V = set_rows(C, set), NW = (int)gridDim.x * 4, npairs = (V + 1) / 2;
  const int cmax = 2 * ((npairs + NW - 1) / NW);
  const int per2 = 2 * cmax;  // pairs per workgroup
  const int total = nsel * per2;
  const unsigned long long* base =
      reinterpret_cast<const unsigned long long*>(C.sam.wlog + (size_t)set * C.sam.wlog_stride);
  constexpr int kB = 8;  // more in flight raises the kernel's registers and slows the head's stream
  for (int e0 = threadIdx.x; e0 < total; e0 += kB * kWG) {
    unsigned long long raw[kB];
    int wg[kB], off[kB];
#pragma unroll
    for (int j = 0; j < kB; j++) {
      const int e = e0 + j * kWG;
      raw[j] = 0ull;
      wg[j] = -1;
      if (e < total) {
        wg[j] = S.sel[e / per2];
        off[j] = e % per2;
        raw[j] = ld_dev_u64(base + (size_t)wg[j] * per2 + off[j]);
      }
    }
#pragma unroll
    for (int j = 0; j < kB; j++) {
      if (wg[j] < 0) continue;
      const int wv = wg[j] * 4 + (2 * off[j]) / cmax, i = (2 * off[j]) % cmax;  // i even
      const int cnt = wv < npairs ? (npairs - 1 - wv) / NW + 1 : 0;
      if (i >= 2 * cnt) continue;
      const int m = 2 * (wv + (i >> 1) * NW);
      const unsigned long long k0 = argmax_key(__uint_as_float((uint32_t)raw[j]), m);
      if (m < V && k0 >= tlo) f(k0);
      if (m + 1 < V) {
        const unsigned long long k1 = argmax_key(__uint_as_float((uint32_t)(raw[j] >> 32)), m + 1);
        if (k1 >= tlo) f(k1);
      }
    }
  }
}

// Top-k distribution of row `set` (0 target, 1 PDM) into S.ids[set] / S.p[set]: the k = min(top_k,
// V) largest logits, value descending (lower index first among equal values), and their softmax at
// temperature 1/inv_temp (max-subtracted, fp32). Whole workgroup; returns k.
__device__ int select_top_k(const Ctx& C, int set, SelLds& S) {
  const int tid = threadIdx.x, lane = tid & 63, G = (int)gridDim.x, V = set_rows(C, set);
  const int k = min(C.sam.top_k, V);
  unsigned long long gm = 0ull;  // G <= kSampleWGs = 4 * kWG: at most four maxima per thread
  {
    unsigned long long x[kSampleWGs / kWG];
#pragma unroll
    for (int j = 0; j < kSampleWGs / kWG; j++) {
      const int i = tid + j * kWG;
      x[j] = i < G ? ld_dev_u64(C.sam.wgmax + (size_t)set * kSampleWGs + i) : 0ull;
    }
#pragma unroll
    for (int j = 0; j < kSampleWGs / kWG; j++) {
      const int i = tid + j * kWG;
      if (i < G) S.keys[i] = x[j];
      gm = x[j] > gm ? x[j] : gm;
    }
  }
  S.gmax[tid] = gm;
  if (tid == 0) {
    S.misc[2] = 0;
    S.misc[3] = 0;
    S.tlo = 1ull;  // every real key is >= 1; stays if fewer than k threads saw a key
  }
  __syncthreads();
  if (gm != 0ull) {  // nonzero values are distinct keys of different vocabulary rows
    int r = 0;
    for (int j = 0; j < kWG; j++) r += S.gmax[j] > gm;
    if (r == k - 1) S.tlo = gm;
  }
  __syncthreads();
  const unsigned long long tlo = S.tlo;
  for (int i = tid; i < G; i += kWG)
    if (S.keys[i] >= tlo) S.sel[atomicAdd(&S.misc[2], 1)] = i;
  __syncthreads();
  const int nsel = S.misc[2];
  visit_regions(C, set, S, nsel, tlo, [&](unsigned long long key) {
    const int at = atomicAdd(&S.misc[3], 1);
    if (at < kSelCap) S.keys[at] = key;
  });
  __syncthreads();
  const int ncand = S.misc[3];  // >= k: every top-k key is a candidate
  if (ncand <= kSelCap) {
    for (int i = tid; i < ncand; i += kWG) {
      const unsigned long long x = S.keys[i];
      int r = 0;
      for (int j = 0; j < ncand; j++) r += S.keys[j] > x;
      if (r < k) {
        S.ids[set][r] = argmax_index(x, V);
        S.p[set][r] = key_value(x);
      }
    }
  } else {
    const unsigned long long T =
        select_kth([&](auto f) { visit_regions(C, set, S, nsel, tlo, f); }, k, S);
    if (tid == 0) S.misc[2] = 0;
    __syncthreads();
    visit_regions(C, set, S, nsel, tlo, [&](unsigned long long key) {
      if (key >= T) {
        const int at = atomicAdd(&S.misc[2], 1);
        if (at < kMaxTopK) S.top[at] = key;
      }
    });
    __syncthreads();
    if (tid < k) {  // exactly k distinct keys are >= T
      const unsigned long long x = S.top[tid];
      int r = 0;
      for (int j = 0; j < k; j++) r += S.top[j] > x;
      S.ids[set][r] = argmax_index(x, V);
      S.p[set][r] = key_value(x);
    }
  }
  __syncthreads();
  if (tid < 64) {  // k <= 64: one wave
    const float top = S.p[set][0];
    const float w = lane < k ? expf((S.p[set][lane] - top) * C.sam.inv_temp) : 0.f;
    const float inv = 1.0f / wave_sum(w);
    if (lane < k) S.p[set][lane] = w * inv;
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

}  // namespace spd
