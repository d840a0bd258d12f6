// GEMV building blocks of the step kernels: a wave multiplies pairs of weight rows by a vector staged
// in LDS, with 16-byte coalesced row loads kept in flight in two alternating register buffers, and a
// fixed per-lane column map, FMA order and butterfly, so that a row's result never depends on which
// wave, workgroup, launch shape or launch mode computes it.
#pragma once
#include "spd_devfn.h"

namespace spd {

// --------------------------------------------------------------------------------------- GEMV
template <typename WT>
__device__ __forceinline__ int gemv_groups(int K) {
  constexpr int BLK = 64 * Elt<WT>::VE;
  return ((K + BLK - 1) / BLK + kU - 1) / kU;
}

// A wave streams NP row pairs against the vector staged in LDS. rowptr(rp, which) returns the first
// element of row `which` of pair rp, or nullptr for a row past the matrix (it contributes zeros).
// The pairs' 16-byte blocks are loaded kU at a time (per row of the pair) into two alternating
// register buffers, so the next group is in flight while the current one is multiplied. Lane rp of
// the wave ends with the pair's two dot products in r0 and r1.
template <typename WT, typename RowFn>
__device__ __forceinline__ void gemv_load(const RowFn& rowptr, int K, int ng, int u, int lane, uint4 (&b)[2][kU]) {
  constexpr int VE = Elt<WT>::VE;
  constexpr int BLK = 64 * VE;
  const int rp = u / ng, g0 = (u - rp * ng) * kU;
  const WT* p0 = rowptr(rp, 0);
  const WT* p1 = rowptr(rp, 1);
#pragma unroll
  for (int uu = 0; uu < kU; uu++) {
    const int col = (g0 + uu) * BLK + lane * VE;
    const bool ok = col < K;  // K is a multiple of VE: a load that starts inside a row ends inside it
    b[0][uu] = (ok && p0 != nullptr) ? ldg16(p0 + col) : make_uint4(0u, 0u, 0u, 0u);
    b[1][uu] = (ok && p1 != nullptr) ? ldg16(p1 + col) : make_uint4(0u, 0u, 0u, 0u);
  }
}

// The FMAs of unit u (the pair's blocks of group gi against the staged vector) into a0, a1.
template <typename WT>
__device__ __forceinline__ void gemv_acc(int nb, int ng, int u, int lane, const float* lds, const uint4 (&b)[2][kU],
                                         float& a0, float& a1) {
  constexpr int VE = Elt<WT>::VE;
  constexpr int BLK = 64 * VE;
  const int rp = u / ng, gi = u - rp * ng, g0 = gi * kU;
  (void)rp;
#pragma unroll
  for (int uu = 0; uu < kU; uu++) {
    const int blk = g0 + uu;
    if (blk < nb) {
      float x[VE];
      const float* xb = lds + blk * BLK;
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
      float w0[VE], w1[VE];
      unpack16<WT>(b[0][uu], w0);
      unpack16<WT>(b[1][uu], w1);
#pragma unroll
      for (int e = 0; e < VE; e++) a0 = fmaf(w0[e], x[e], a0);
#pragma unroll
      for (int e = 0; e < VE; e++) a1 = fmaf(w1[e], x[e], a1);
    }
  }
}

// After unit u's FMAs: if it was the pair's last group, reduce across the wave (fixed butterfly) and
// hand the pair's two dot products to done.
template <typename DoneFn>
__device__ __forceinline__ void gemv_fin(int ng, int u, float& a0, float& a1, const DoneFn& done) {
  const int rp = u / ng, gi = u - rp * ng;
  if (gi == ng - 1) {
    const float s0 = wave_sum(a0), s1 = wave_sum(a1);
    done(rp, s0, s1);
    a0 = 0.f;
    a1 = 0.f;
  }
}

// A wave streams `count` row pairs against the vector staged in LDS: pair i of the wave is
// rowptr(i, 0) and rowptr(i, 1) (nullptr rows contribute zeros), and when its two dot products are
// reduced every lane calls done(i, s0, s1). The units (pair, group of kU blocks) are loaded two ahead
// into the alternating buffers, across pair boundaries, so a wave's loads never stop between pairs;
// stream_prefetch requests the first two before the vector is staged.
template <typename WT, typename RowFn>
__device__ __forceinline__ void stream_prefetch(const RowFn& rowptr, int count, int K, int lane, uint4 (&bA)[2][kU],
                                                uint4 (&bB)[2][kU]) {
  const int ng = gemv_groups<WT>(K);
  if (count * ng > 0) gemv_load<WT>(rowptr, K, ng, 0, lane, bA);
  if (count * ng > 1) gemv_load<WT>(rowptr, K, ng, 1, lane, bB);
}

template <typename WT, typename RowFn, typename DoneFn>
__device__ __forceinline__ void stream_run(const RowFn& rowptr, const DoneFn& done, int count, int K, int lane,
                                           const float* lds, uint4 (&bA)[2][kU], uint4 (&bB)[2][kU]) {
  constexpr int BLK = 64 * Elt<WT>::VE;
  const int nb = (K + BLK - 1) / BLK;
  const int ng = (nb + kU - 1) / kU;
  const int NU = count * ng;
  float a0 = 0.f, a1 = 0.f;
  // each buffer is refilled as soon as its unit's FMAs have read it, before that unit's reduction and
  // epilogue (whose stores the compiler would otherwise keep ahead of the next loads)
  for (int u = 0; u < NU; u += 2) {
    gemv_acc<WT>(nb, ng, u, lane, lds, bA, a0, a1);
    if (u + 2 < NU) gemv_load<WT>(rowptr, K, ng, u + 2, lane, bA);
    gemv_fin(ng, u, a0, a1, done);
    if (u + 1 < NU) {
      gemv_acc<WT>(nb, ng, u + 1, lane, lds, bB, a0, a1);
      if (u + 3 < NU) gemv_load<WT>(rowptr, K, ng, u + 3, lane, bB);
      gemv_fin(ng, u + 1, a0, a1, done);
    }
  }
}


// Several rows against the same weights: a wave streams its row pairs once and multiplies every
// block by the nr (<= NR) vectors staged in LDS (vector r at lds + r * ldsK), each row keeping its
// own accumulators in the single-row FMA order; when a pair's last group is done every lane calls
// done(pair, s0, s1) with the nr rows' two dot products (entries >= nr are zero).
template <typename WT, int NR>
__device__ __forceinline__ void rgemv_acc(int nb, int ng, int u, int lane, const float* lds, int ldsK, int nr,
                                          const uint4 (&b)[2][kU], float (&a0)[NR], float (&a1)[NR]) {
  constexpr int VE = Elt<WT>::VE;
  constexpr int BLK = 64 * VE;
  const int gi = u % ng, g0 = gi * kU;
#pragma unroll
  for (int uu = 0; uu < kU; uu++) {
    const int blk = g0 + uu;
    if (blk < nb) {
      float w0[VE], w1[VE];
      unpack16<WT>(b[0][uu], w0);
      unpack16<WT>(b[1][uu], w1);
#pragma unroll
      for (int r = 0; r < NR; r++) {
        if (r < nr) {
          float x[VE];
          const float* xb = lds + (size_t)r * ldsK + blk * BLK;
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
          for (int e = 0; e < VE; e++) a0[r] = fmaf(w0[e], x[e], a0[r]);
#pragma unroll
          for (int e = 0; e < VE; e++) a1[r] = fmaf(w1[e], x[e], a1[r]);
        }
      }
    }
  }
}

template <int NR, typename DoneFn>
__device__ __forceinline__ void rgemv_fin(int ng, int u, int nr, float (&a0)[NR], float (&a1)[NR], const DoneFn& done) {
  const int rp = u / ng, gi = u - rp * ng;
  if (gi == ng - 1) {
    float s0[NR], s1[NR];
#pragma unroll
    for (int r = 0; r < NR; r++) {
      s0[r] = r < nr ? wave_sum(a0[r]) : 0.f;
      s1[r] = r < nr ? wave_sum(a1[r]) : 0.f;
      a0[r] = 0.f;
      a1[r] = 0.f;
    }
    done(rp, s0, s1);
  }
}

template <typename WT, int NR, typename RowFn, typename DoneFn>
__device__ __forceinline__ void rstream_run(const RowFn& rowptr, const DoneFn& done, int count, int K, int lane,
                                            const float* lds, int ldsK, int nr, uint4 (&bA)[2][kU],
                                            uint4 (&bB)[2][kU]) {
  constexpr int BLK = 64 * Elt<WT>::VE;
  const int nb = (K + BLK - 1) / BLK;
  const int ng = (nb + kU - 1) / kU;
  const int NU = count * ng;
  float a0[NR], a1[NR];
#pragma unroll
  for (int r = 0; r < NR; r++) a0[r] = a1[r] = 0.f;
  for (int u = 0; u < NU; u += 2) {
    rgemv_acc<WT, NR>(nb, ng, u, lane, lds, ldsK, nr, bA, a0, a1);
    if (u + 2 < NU) gemv_load<WT>(rowptr, K, ng, u + 2, lane, bA);
    rgemv_fin<NR>(ng, u, nr, a0, a1, done);
    if (u + 1 < NU) {
      rgemv_acc<WT, NR>(nb, ng, u + 1, lane, lds, ldsK, nr, bB, a0, a1);
      if (u + 3 < NU) gemv_load<WT>(rowptr, K, ng, u + 3, lane, bB);
      rgemv_fin<NR>(ng, u + 1, nr, a0, a1, done);
    }
  }
}

// Stage src[0, K) into LDS in the xidx layout, zero padded to the block multiple, times gain[k] when a
// gain is given. Returns the workgroup's sum of squares of src when a
// gain is given: each thread sums its float4 groups in the same order as the per-sublayer kernels'
// staging, then the fixed block reduction, so both launch modes compute the same norm bit for bit.
// Ends with a barrier, so the vector is visible to all waves.
template <int VE>
__device__ __forceinline__ float stage_vec(const float* src, const float* gain, int K, float* lds, float* red) {
  constexpr int BLK = 64 * VE;
  constexpr int RND = 4;
  const int n4 = ((K + BLK - 1) / BLK * BLK) >> 2;
  float ss = 0.f;
  for (int k40 = threadIdx.x; k40 < n4; k40 += kWG * RND) {
    float4 v[RND], g[RND];
#pragma unroll
    for (int j = 0; j < RND; j++) {
      const int k = (k40 + j * kWG) * 4;
      const bool ok = k < K;  // K is a multiple of 4
      if (ok) {
        v[j] = *reinterpret_cast<const float4*>(src + k);
      } else {
        v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      }
      g[j] = (ok && gain != nullptr) ? *reinterpret_cast<const float4*>(gain + k) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
#pragma unroll
    for (int j = 0; j < RND; j++) {
      const int k4 = k40 + j * kWG;
      if (k4 < n4) {
        float4 val = v[j];
        if (gain != nullptr) {
          ss = fmaf(val.x, val.x, ss);
          ss = fmaf(val.y, val.y, ss);
          ss = fmaf(val.z, val.z, ss);
          ss = fmaf(val.w, val.w, ss);
          val.x *= g[j].x;
          val.y *= g[j].y;
          val.z *= g[j].z;
          val.w *= g[j].w;
        }
        *reinterpret_cast<float4*>(lds + xidx<VE>(k4 * 4)) = val;
      }
    }
  }
  if (gain != nullptr) return block_sum(ss, red);
  __syncthreads();
  return 0.f;
}


}  // namespace spd
