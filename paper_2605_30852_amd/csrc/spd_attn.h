// Decode attention of one token over one KV head's paged cache, one key split per workgroup (the
// stage launches and the row-block launches share it, so both compute the same bits).
//
// The token at position pos0 attends to keys 0..pos0 of its own layer (Section 3.1: each stage's
// token reads the cache of the layer it is on). Its G query heads share KV head g (grouped-query
// attention). A split covers keys [k0, k1) in rounds of 64 keys, 16 per wave, and the waves never
// wait for each other inside the split:
//   * lane l of a wave owns key l/4 of the wave's 16 and a quarter of the head dimension, for K and V
//     alike (one page-table lookup serves both); a round's loads are issued two rounds ahead and the
//     page of the round after is requested before them, so no wait for a page ever waits for K or V;
//   * scores are dot products over the quarter, summed across the four lanes of a key with DPP; the
//     lanes of a key then split the heads between them (head h on lane h mod 4), so the online
//     softmax of a head is a 16-lane max and sum;
//   * P.V goes through a wave-private LDS tile: lane l accumulates one head's slice of dimensions over
//     the wave's keys in key order.
// Each wave keeps its own running (m, l, o); the four are combined in wave order at the end of the
// split (one barrier). With one split the workgroup writes the output; otherwise the split that
// finishes last (a ticket per stage and head) merges every split in split order, its loads for up to
// 32 splits issued at once. The split size is a function of the configuration only, so a token's
// result never depends on how many stages run.
#pragma once
#include "spd_devfn.h"

namespace spd {

constexpr int kAttnTPK = 4;                   // lanes per key
constexpr int kAttnWaveKeys = 64 / kAttnTPK;  // keys per wave per round
constexpr int kAttnPass = kWG / kAttnTPK;     // keys per round
constexpr int kAttnMaxQ = 8;                  // query heads per KV head
constexpr int kAttnMergeBatch = 32;           // splits whose partial outputs the merge loads at once

// LDS: pre-scaled queries, then per wave a V tile (reused for the wave's o at the end), its
// probabilities, and its rescale factors and (m, l).
template <typename KVT, int DH>
struct AttnLds {
  static constexpr int kWaves = kWG / 64;
  static constexpr size_t kQ = (size_t)kAttnMaxQ * DH * 4;
  static constexpr size_t kTile = (size_t)kAttnWaveKeys * DH * sizeof(KVT);
  static constexpr size_t kO = (size_t)kAttnMaxQ * DH * 4;
  static constexpr size_t kVt = kTile > kO ? kTile : kO;
  static constexpr size_t kP = (size_t)kAttnMaxQ * kAttnWaveKeys * 4;
  static constexpr size_t kA = (size_t)kAttnMaxQ * 4 * 3;  // alpha, m, l
  static constexpr size_t kWave = kVt + kP + kA;
  static constexpr size_t kTotal = kQ + kWaves * kWave;
};

template <typename KVT, int DH>
constexpr size_t attn_split_lds() {
  return AttnLds<KVT, DH>::kTotal;
}

// KV cache reads. Ordinary loads: a round's keys come back faster than with the non-temporal hint.
__device__ __forceinline__ uint4 ldkv16(const void* p) { return *reinterpret_cast<const uint4*>(p); }

__device__ __forceinline__ void st_dev2f(float* p, float x, float y) {  // p 8-byte aligned
  const unsigned long long u = (unsigned long long)__float_as_uint(x) | ((unsigned long long)__float_as_uint(y) << 32);
  __hip_atomic_store((unsigned long long*)p, u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Sum over the four lanes of a quad (DPP quad permutes); all four lanes get the same bits.
__device__ __forceinline__ float quad_sum(float v) {
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xB1, 0xF, 0xF, false));  // lane ^ 1
  v += __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x4E, 0xF, 0xF, false));  // lane ^ 2
  return v;
}

// Max / sum over the 16 lanes of a wave that share lane mod 4; every such lane gets the same bits.
__device__ __forceinline__ float key_max(float v) {
#pragma unroll
  for (int m = 4; m < 64; m <<= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}
__device__ __forceinline__ float key_sum(float v) {
#pragma unroll
  for (int m = 4; m < 64; m <<= 1) v += __shfl_xor(v, m, 64);
  return v;
}

// Orders the wave's LDS writes before its later LDS reads of other lanes' data (one wave executes
// its LDS operations in order; this keeps the compiler from moving them).
__device__ __forceinline__ void wave_lds_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// N consecutive KV elements from LDS as floats (N * sizeof(T): 8 bytes or a multiple of 16, aligned).
template <typename T, int N>
__device__ __forceinline__ void lds_row(const T* p, float* o) {
  constexpr int BYTES = N * (int)sizeof(T);
  if constexpr (BYTES % 16 == 0) {
#pragma unroll
    for (int c = 0; c < BYTES / 16; c++)
      unpack16<T>(reinterpret_cast<const uint4*>(p)[c], o + c * (16 / (int)sizeof(T)));
  } else {
    static_assert(BYTES == 8, "row of 8 bytes or a multiple of 16");
    const uint2 u = *reinterpret_cast<const uint2*>(p);
    if constexpr (sizeof(T) == 2) {
      o[0] = bf_lo(u.x);
      o[1] = bf_hi(u.x);
      o[2] = bf_lo(u.y);
      o[3] = bf_hi(u.y);
    } else {
      o[0] = __uint_as_float(u.x);
      o[1] = __uint_as_float(u.y);
    }
  }
}

// Merge of one (token, KV head)'s nsplit split records (o[8][DH], m[8], l[8]; every split has a key,
// so each m is finite) in split order into its G output rows. Every thread of the workgroup calls it.
// All (m, l) pairs are requested first, then the first batch of partial outputs (only the entries
// that exist: the records are read past the L2, where a repeated address costs as much as a new
// one), then the (m, l) pairs go to LDS (sm: 2 * kMaxSplits * kAttnMaxQ floats).
template <int DH>
__device__ __forceinline__ void attn_merge(const float* rec_base, int nsplit, int G, float* out, float* sm) {
  constexpr int MAXQ = kAttnMaxQ, RS = MAXQ * (DH + 2);
  constexpr int NPAIR = MAXQ * DH / 2;
  constexpr int PPT = (NPAIR + kWG - 1) / kWG;
  const int tid = threadIdx.x;
  constexpr int MB = kAttnMergeBatch;
  constexpr int MLT = (kMaxSplits * MAXQ + kWG - 1) / kWG;
  float* sl = sm + kMaxSplits * MAXQ;
  float mlm[MLT], mll[MLT];
#pragma unroll
  for (int i = 0; i < MLT; i++) {
    const int t = tid + i * kWG, sp = t / G, qi = t % G;
    mlm[i] = mll[i] = 0.f;
    if (t < nsplit * G) {
      mlm[i] = ld_dev(rec_base + (size_t)sp * RS + MAXQ * DH + qi);
      mll[i] = ld_dev(rec_base + (size_t)sp * RS + MAXQ * DH + MAXQ + qi);
    }
  }
  const int qi0 = tid / (DH / 2), dp0 = tid % (DH / 2);
  const int qc0 = min(qi0, G - 1);
  float2 ob[MB];
#pragma unroll
  for (int j = 0; j < MB; j++)
    ob[j] = (j < nsplit && qi0 < G) ? ld_dev2(rec_base + (size_t)j * RS + qc0 * DH + 2 * dp0) : make_float2(0.f, 0.f);
#pragma unroll
  for (int i = 0; i < MLT; i++) {
    const int t = tid + i * kWG;
    if (t < nsplit * G) {
      sm[(t / G) * MAXQ + t % G] = mlm[i];
      sl[(t / G) * MAXQ + t % G] = mll[i];
    }
  }
  __syncthreads();
#pragma unroll 1
  for (int i = 0; i < PPT; i++) {
    const int e = tid + i * kWG, qi = e / (DH / 2), dp = e % (DH / 2);
    if (qi < G) {
      float M = -INFINITY;
      for (int sp = 0; sp < nsplit; sp++) M = fmaxf(M, sm[sp * MAXQ + qi]);
      float L = 0.f, a0 = 0.f, a1 = 0.f;
      for (int sp0 = 0; sp0 < nsplit; sp0 += MB) {
        if (i > 0 || sp0 > 0) {
#pragma unroll
          for (int j = 0; j < MB; j++)
            ob[j] = ld_dev2(rec_base + (size_t)min(sp0 + j, nsplit - 1) * RS + qi * DH + 2 * dp);
        }
#pragma unroll
        for (int j = 0; j < MB; j++) {
          if (sp0 + j < nsplit) {
            const float f = expf(sm[(sp0 + j) * MAXQ + qi] - M);
            L = fmaf(sl[(sp0 + j) * MAXQ + qi], f, L);
            a0 = fmaf(ob[j].x, f, a0);
            a1 = fmaf(ob[j].y, f, a1);
          }
        }
      }
      const float inv = 1.0f / L;
      *reinterpret_cast<float2*>(out + qi * DH + 2 * dp) = make_float2(a0 * inv, a1 * inv);
    }
  }
}

// One split with GP head slots (4: G <= 4, 8: G <= 8). Arguments as for attn_split.
template <typename KVT, int DH, int GP>
__device__ bool attn_split_g(const Ctx& C, const KVT* kvb, const float* q, float* out, float* rec_base, int* cnt,
                             int g, int split, int nsplit, int k0, int k1, int pos0, int page0, float* lds) {
  constexpr int TPK = kAttnTPK, NE = DH / TPK, VE = Elt<KVT>::VE, KCH = NE / VE;
  constexpr int WK = kAttnWaveKeys, PASS = kAttnPass, MAXQ = kAttnMaxQ, NJ = GP / 4;
  constexpr int LPH = 64 / GP, DPL = DH / LPH;  // P.V: lanes per head, dimensions per lane
  constexpr int KUNR = DPL > 8 ? 2 : 4;          // P.V keys in flight
  constexpr int RS = MAXQ * (DH + 2);
  using LA = AttnLds<KVT, DH>;
  __shared__ int s_last;
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int kk = lane / TPK, qq = lane % TPK;
  const int G = C.G;
  char* const lbase = reinterpret_cast<char*>(lds);
  float* qs = lds;                                                  // [MAXQ][DH] pre-scaled queries
  char* wbase = lbase + LA::kQ + (size_t)w * LA::kWave;
  KVT* vt = reinterpret_cast<KVT*>(wbase);                          // [WK][DH] V tile, then o [MAXQ][DH]
  float* pt = reinterpret_cast<float*>(wbase + LA::kVt);            // [MAXQ][WK] probabilities
  float* at = reinterpret_cast<float*>(wbase + LA::kVt + LA::kP);   // alpha[MAXQ], m[MAXQ], l[MAXQ]
  const size_t page_elems = (size_t)2 * C.hkv * C.page * DH;
  const size_t head_off = (size_t)g * C.page * DH;
  const size_t voff = (size_t)C.hkv * C.page * DH;
  const int R = (k1 - k0 + PASS - 1) / PASS;  // rounds
  const int my = w * WK + kk;                 // this lane's key within a round

  // Every global load below is unconditional (keys past the split read the slot of key k1 - 1, in
  // round 0 of the page their own key falls in, and are masked later), so the count of loads issued after any given load is the same on every path and each
  // wait covers exactly the loads it needs: queries first, then the page of round 1, round 0, the
  // page of round 2, round 1.
  constexpr int QPT = (MAXQ * DH + kWG - 1) / kWG;
  float qv[QPT];
#pragma unroll
  for (int i = 0; i < QPT; i++) {
    const int e = min(tid + i * kWG, G * DH - 1);
    qv[i] = q[e];
  }
  auto page_of = [&](int r) { return C.page_table[min(k0 + r * PASS + my, k1 - 1) / C.page]; };
  int pg_next = page_of(1);
  uint4 kb0[KCH], vb0[KCH], kb1[KCH], vb1[KCH];
  auto issue = [&](int r, int page, uint4* kr, uint4* vr) {
    const int key = min(k0 + r * PASS + my, k1 - 1);
    const KVT* base = kvb + (size_t)page * page_elems + head_off + (size_t)(key % C.page) * DH + qq * NE;
#pragma unroll
    for (int c = 0; c < KCH; c++) kr[c] = ldkv16(reinterpret_cast<const uint4*>(base) + c);
#pragma unroll
    for (int c = 0; c < KCH; c++) vr[c] = ldkv16(reinterpret_cast<const uint4*>(base + voff) + c);
  };
  issue(0, page0, kb0, vb0);
  {
    const int pg1 = pg_next;
    pg_next = page_of(2);
    issue(1, pg1, kb1, vb1);
  }
#pragma unroll
  for (int i = 0; i < QPT; i++) qs[tid + i * kWG] = qv[i] * C.scale;  // slots >= G: unused
  __syncthreads();  // queries staged

  float m_run[NJ], l_run[NJ];
#pragma unroll
  for (int j = 0; j < NJ; j++) {
    m_run[j] = -INFINITY;
    l_run[j] = 0.f;
  }
  const int ph = lane / LPH, pd = (lane % LPH) * DPL;  // P.V: head slot and first dimension
  float o[DPL];
#pragma unroll
  for (int e = 0; e < DPL; e++) o[e] = 0.f;

  auto round = [&](int r, uint4* kr_raw, uint4* vr_raw) {
    const int kbase = k0 + r * PASS + w * WK;  // the wave's first key in this round
    const int nkw = min(WK, k1 - kbase);       // wave-uniform
    float kf[NE];
#pragma unroll
    for (int c = 0; c < KCH; c++) unpack16<KVT>(kr_raw[c], kf + c * VE);
    // a key past the end may come from a page beyond the cache's length (round 0's page is looked up
    // before the length is known), whose contents are arbitrary: its V row enters the tile as zeros,
    // so that its zero probability keeps the sums exact even if those bytes are not a finite number
    const bool kin = kk < nkw;
#pragma unroll
    for (int c = 0; c < KCH; c++)
      reinterpret_cast<uint4*>(vt + kk * DH + qq * NE)[c] = kin ? vr_raw[c] : make_uint4(0u, 0u, 0u, 0u);
    {  // the buffers are free again: round r + 2, and the page of round r + 3 (past the end: key k1 - 1)
      const int pg = pg_next;
      pg_next = page_of(r + 3);
      issue(r + 2, pg, kr_raw, vr_raw);
    }
    if (nkw > 0) {  // else the wave has no key in this round
      const bool valid = kk < nkw;
      float sel[NJ];
#pragma unroll
      for (int j = 0; j < NJ; j++) sel[j] = -INFINITY;
#pragma unroll
      for (int qi = 0; qi < GP; qi++) {
        if (qi < G) {
          const float* qp = qs + qi * DH + qq * NE;
          float dsum = 0.f;
#pragma unroll
          for (int e = 0; e < NE; e += 4) {
            const float4 q4 = *reinterpret_cast<const float4*>(qp + e);
            dsum = fmaf(q4.x, kf[e], dsum);
            dsum = fmaf(q4.y, kf[e + 1], dsum);
            dsum = fmaf(q4.z, kf[e + 2], dsum);
            dsum = fmaf(q4.w, kf[e + 3], dsum);
          }
          dsum = quad_sum(dsum);
          if ((qi & 3) == qq) sel[qi >> 2] = valid ? dsum : -INFINITY;
        }
      }
      // online softmax of head qq + 4j over the wave's keys (key 0 of the round is valid, so mn is
      // finite for every head h < G)
#pragma unroll
      for (int j = 0; j < NJ; j++) {
        const int h = qq + 4 * j;
        const float mx = key_max(sel[j]);
        const float mn = fmaxf(m_run[j], mx);
        const float al = m_run[j] == -INFINITY ? 0.f : expf(m_run[j] - mn);
        const float p = valid && h < G ? expf(sel[j] - mn) : 0.f;
        const float ps = key_sum(p);
        l_run[j] = l_run[j] * al + ps;
        m_run[j] = mn;
        if (h < G) {
          pt[h * WK + kk] = p;
          if (kk == 0) at[h] = al;
        }
      }
      wave_lds_sync();
      if (ph < G) {
        const float al = at[ph];
#pragma unroll
        for (int e = 0; e < DPL; e++) o[e] *= al;
        const float* pp = pt + ph * WK;
#pragma unroll KUNR
        for (int k = 0; k < WK; k++) {
          float v[DPL];
          lds_row<KVT, DPL>(vt + k * DH + pd, v);
          const float pk = pp[k];
#pragma unroll
          for (int e = 0; e < DPL; e++) o[e] = fmaf(pk, v[e], o[e]);
        }
      }
    }
    wave_lds_sync();  // the tile and probabilities are rewritten next round
  };
  for (int r = 0; r < R; r += 2) {  // an odd count ends with a round that has no key
    round(r, kb0, vb0);
    round(r + 1, kb1, vb1);
  }

  // the wave's (m, l, o) to LDS; o reuses the V tile
  float* ow = reinterpret_cast<float*>(vt);
#pragma unroll
  for (int j = 0; j < NJ; j++) {
    const int h = qq + 4 * j;
    if (kk == 0 && h < G) {
      at[MAXQ + h] = m_run[j];
      at[2 * MAXQ + h] = l_run[j];
    }
  }
  if (ph < G) {
#pragma unroll
    for (int e = 0; e < DPL; e++) ow[ph * DH + pd + e] = o[e];
  }
  __syncthreads();

  // combine the waves in wave order: (A, M, L) of the split per (head, dimension pair); a wave with
  // no key has m = -inf and weight 0 (wave 0 always has key k0, so M is finite)
  constexpr int NW = LA::kWaves;
  constexpr int NPAIR = MAXQ * DH / 2;
  constexpr int PPT = (NPAIR + kWG - 1) / kWG;
  float A0[PPT], A1[PPT], Ms[PPT], Ls[PPT];
#pragma unroll
  for (int i = 0; i < PPT; i++) {
    const int e = tid + i * kWG, qi = e / (DH / 2), dp = e % (DH / 2);
    A0[i] = A1[i] = Ms[i] = Ls[i] = 0.f;
    if (qi < G) {
      float M = -INFINITY;
#pragma unroll
      for (int wv = 0; wv < NW; wv++)
        M = fmaxf(M, reinterpret_cast<const float*>(lbase + LA::kQ + (size_t)wv * LA::kWave + LA::kVt + LA::kP)[MAXQ + qi]);
      float L = 0.f, a0 = 0.f, a1 = 0.f;
#pragma unroll
      for (int wv = 0; wv < NW; wv++) {
        const char* wb = lbase + LA::kQ + (size_t)wv * LA::kWave;
        const float* aw = reinterpret_cast<const float*>(wb + LA::kVt + LA::kP);
        const float mw = aw[MAXQ + qi];
        if (mw != -INFINITY) {
          const float f = expf(mw - M);
          L = fmaf(aw[2 * MAXQ + qi], f, L);
          const float2 ov = *reinterpret_cast<const float2*>(reinterpret_cast<const float*>(wb) + qi * DH + 2 * dp);
          a0 = fmaf(ov.x, f, a0);
          a1 = fmaf(ov.y, f, a1);
        }
      }
      A0[i] = a0;
      A1[i] = a1;
      Ms[i] = M;
      Ls[i] = L;
    }
  }
  if (nsplit == 1) {
#pragma unroll
    for (int i = 0; i < PPT; i++) {
      const int e = tid + i * kWG, qi = e / (DH / 2), dp = e % (DH / 2);
      if (qi < G) {
        const float inv = 1.0f / Ls[i];
        *reinterpret_cast<float2*>(out + qi * DH + 2 * dp) = make_float2(A0[i] * inv, A1[i] * inv);
      }
    }
    return true;
  }
  float* rec = rec_base + (size_t)split * RS;
#pragma unroll
  for (int i = 0; i < PPT; i++) {
    const int e = tid + i * kWG, qi = e / (DH / 2), dp = e % (DH / 2);
    if (qi < G) {
      st_dev2f(rec + qi * DH + 2 * dp, A0[i], A1[i]);
      if (dp == 0) {
        st_dev(rec + MAXQ * DH + qi, Ms[i]);
        st_dev(rec + MAXQ * DH + MAXQ + qi, Ls[i]);
      }
    }
  }
  wait_own_stores();
  __syncthreads();
  if (tid == 0) {
    const int t = __hip_atomic_fetch_add(cnt, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    s_last = (t == nsplit - 1);
  }
  __syncthreads();
  if (!s_last) return false;

  attn_merge<DH>(rec_base, nsplit, G, out, reinterpret_cast<float*>(lbase + LA::kQ));
  if (tid == 0) __hip_atomic_store(cnt, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return true;
}

// ------------------------------------------------------------- row blocks on matrix cores
// A row block's rows sit at consecutive positions pos0 .. pos0 + nrows - 1 and all read one cache (the
// draft module's in-flight rows over its KV, Eq. input-seq; a prefill chunk over the prompt), row r's G
// query heads attending keys 0 .. pos0 + r (causal). One pass over a key split of KV head g then
// serves all nrows * G <= 32 queries (query j = r * G + h) as the columns of 32x32 fp32 MFMA tiles
// (v_mfma_f32_32x32x2f32: lane l supplies A[l%32][l/32] and B[l/32][l%32]; accumulator register v of
// lane l is row 8(v/4) + 4(l/32) + v%4, column l%32). Each wave takes 32-key tiles of the split:
//   * S^T = K Q^T: k-step kc contracts dims kc and DH/2 + kc, so lane l needs dims (l/32)*DH/2 ..
//     + DH/2 of key l%32 (one contiguous run, loaded once) and of query l%32 (registers); lane l then
//     holds query l%32's scores of keys 8(v/4) + 4(l/32) + v%4;
//   * online softmax per query: a max and a sum over the lane's 16 scores and one exchange with lane
//     l ^ 32, which holds the query's other 16;
//   * O^T += V^T P^T: k-step v contracts the two keys of register v, whose probabilities the lanes
//     already hold as their B operand; A is V^T with row i of dim tile t standing for dim
//     i * DH/32 + t, so a lane reads the DH/32 values of all tiles as one run of its V row (staged in
//     a wave-private LDS tile). Lane l ends with query l%32's output over its 16 rows per tile.
// The products are exact (fp32 operands, fp32 accumulation); against the one-token split only the
// order of the sums differs. The four waves' (m, l, o) combine in wave order; a row with one split
// writes its output, otherwise its split record (the one-token split's layout and ticket per row and
// KV head), and the workgroup that finishes a row's last split merges it in split order.
typedef float mfma_acc16 __attribute__((ext_vector_type(16)));

template <int DH>
struct RowsMfmaLds {
  static constexpr int kWaves = kWG / 64;
  static constexpr size_t kRow = (size_t)DH * 2 + 16;                 // bf16 V row + pad (banks)
  static constexpr size_t kVTiles = (size_t)kWaves * 32 * kRow;       // per wave [32 keys][DH]
  static constexpr size_t kO = (size_t)kWaves * 32 * DH * 4;          // per wave o[32 queries][DH]
  static constexpr size_t kMain = kVTiles > kO ? kVTiles : kO;
  static constexpr size_t kML = (size_t)kWaves * 32 * 2 * 4;          // per wave m[32], l[32]
  static constexpr size_t kMerge = (size_t)2 * kMaxSplits * kAttnMaxQ * 4;
  static constexpr size_t kTotal = kMain + kML + (kMerge > kMain ? kMerge - kMain : 0);
};

template <int DH>
constexpr size_t attn_rows_mfma_lds() {
  return RowsMfmaLds<DH>::kTotal;
}

// bf16 element e of a run of packed bf16 words, as fp32 (exact)
template <int N>
__device__ __forceinline__ float bf_at(const uint4 (&w)[N], int e) {
  const uint4 v = w[e >> 3];
  const int k = (e >> 1) & 3;
  const uint32_t u = k == 0 ? v.x : k == 1 ? v.y : k == 2 ? v.z : v.w;
  return (e & 1) ? bf_hi(u) : bf_lo(u);
}

// One key split [k0, k0 + chunk) of KV head g for the rows of a block. kvb: the layer's bf16 cache;
// q, out: the block's query and output rows (row r at r * qdim, head g's G heads contiguous);
// part, cnt: the split records and tickets of (row r, KV head g) at index r * hkv + g.
template <int DH>
__device__ void attn_rows_mfma(const Ctx& C, const uint16_t* kvb, const float* q, float* out, float* part, int* cnt,
                               int g, int split, int nrows, int pos0, float* lds) {
  constexpr int HALF = DH / 2, NT = DH / 32, KV16 = HALF / 8;  // dims per lane half, dim tiles, uint4 per run
  constexpr int MAXQ = kAttnMaxQ, RS = MAXQ * (DH + 2);
  using LA = RowsMfmaLds<DH>;
  __shared__ int s_last[kMaxRows];
  const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63;
  const int col = lane & 31, hf = lane >> 5;
  const int G = C.G, M = nrows * G;
  const int kend = pos0 + nrows;  // keys of the block: [0, kend)
  const int k0 = split * C.chunk, k1 = min(kend, k0 + C.chunk);
  char* const lbase = reinterpret_cast<char*>(lds);
  char* const vt = lbase + (size_t)w * 32 * LA::kRow;  // this wave's V tile
  const size_t page_elems = (size_t)2 * C.hkv * C.page * DH;
  const size_t head_off = (size_t)g * C.page * DH;
  const size_t voff = (size_t)C.hkv * C.page * DH;

  // this lane's query: column col; row r = col / G, head h = col % G (columns >= M are zero)
  const int qr = col / G, qh = col % G;
  const bool qon = col < M;
  const int qlim = pos0 + qr;  // last key the query attends
  float qf[HALF];
  {
    const float* qp = q + (size_t)min(qr, nrows - 1) * C.qdim + (size_t)(g * G + qh) * DH + hf * HALF;
#pragma unroll
    for (int e = 0; e < HALF; e += 4) {
      const float4 v = *reinterpret_cast<const float4*>(qp + e);
      qf[e] = qon ? v.x * C.scale : 0.f;
      qf[e + 1] = qon ? v.y * C.scale : 0.f;
      qf[e + 2] = qon ? v.z * C.scale : 0.f;
      qf[e + 3] = qon ? v.w * C.scale : 0.f;
    }
  }
  const int ntiles = (k1 - k0 + 31) / 32;
  auto key_of = [&](int t) { return min(k0 + t * 32 + col, k1 - 1); };  // this lane's key of tile t (clamped)
  uint4 kr[KV16], vr[KV16];
  auto issue = [&](int t, int page) {
    const int key = key_of(t);
    const uint16_t* base = kvb + (size_t)page * page_elems + head_off + (size_t)(key % C.page) * DH + hf * HALF;
#pragma unroll
    for (int c = 0; c < KV16; c++) kr[c] = ldkv16(reinterpret_cast<const uint4*>(base) + c);
#pragma unroll
    for (int c = 0; c < KV16; c++) vr[c] = ldkv16(reinterpret_cast<const uint4*>(base + voff) + c);
  };
  // every wave runs the same number of tile steps (a step past the split's tiles loads the last key
  // and masks everything), so the MFMAs always run on full waves
  const int steps = (ntiles + LA::kWaves - 1) / LA::kWaves;
  int t = w;
  int pg_next = C.page_table[key_of(min(t + LA::kWaves, ntiles - 1)) / C.page];
  issue(min(t, ntiles - 1), C.page_table[key_of(min(t, ntiles - 1)) / C.page]);

  float m_run = -INFINITY, l_run = 0.f;
  mfma_acc16 o[NT];
#pragma unroll
  for (int tt = 0; tt < NT; tt++)
#pragma unroll
    for (int v = 0; v < 16; v++) o[tt][v] = 0.f;

  for (int it = 0; it < steps; it++, t += LA::kWaves) {
    const int kb = k0 + t * 32;  // the tile's first key (t past the end: nothing valid)
    // V run of key col to the wave's tile
#pragma unroll
    for (int c = 0; c < KV16; c++) reinterpret_cast<uint4*>(vt + (size_t)col * LA::kRow + hf * HALF * 2)[c] = vr[c];
    mfma_acc16 sacc;
#pragma unroll
    for (int v = 0; v < 16; v++) sacc[v] = 0.f;
#pragma unroll
    for (int kc = 0; kc < HALF; kc++) sacc = __builtin_amdgcn_mfma_f32_32x32x2f32(bf_at(kr, kc), qf[kc], sacc, 0, 0, 0);
    {  // the registers are free again: the next tile, and the page of the one after
      const int tn = min(t + LA::kWaves, ntiles - 1);
      const int pg = pg_next;
      pg_next = C.page_table[key_of(min(t + 2 * LA::kWaves, ntiles - 1)) / C.page];
      issue(tn, pg);
    }
    float p[16];
    float mx = -INFINITY;
#pragma unroll
    for (int v = 0; v < 16; v++) {
      const int key = kb + 8 * (v >> 2) + 4 * hf + (v & 3);
      const bool ok = qon && t < ntiles && key < k1 && key <= qlim;
      p[v] = ok ? sacc[v] : -INFINITY;
      mx = fmaxf(mx, p[v]);
    }
    mx = fmaxf(mx, __shfl_xor(mx, 32, 64));
    const float mn = fmaxf(m_run, mx);
    const float al = m_run == -INFINITY ? 0.f : expf(m_run - mn);
    float ps = 0.f;
#pragma unroll
    for (int v = 0; v < 16; v++) {
      p[v] = p[v] == -INFINITY ? 0.f : expf(p[v] - mn);
      ps += p[v];
    }
    ps += __shfl_xor(ps, 32, 64);
    l_run = l_run * al + ps;
    m_run = mn;
#pragma unroll
    for (int tt = 0; tt < NT; tt++)
#pragma unroll
      for (int v = 0; v < 16; v++) o[tt][v] *= al;
    wave_lds_sync();  // the V tile is written
#pragma unroll
    for (int v = 0; v < 16; v++) {
      const int kr_ = 8 * (v >> 2) + 4 * hf + (v & 3);  // the key of register v on this lane half
      const char* vp = vt + (size_t)kr_ * LA::kRow + col * NT * 2;
      float a[NT];
      if constexpr (NT == 4) {
        const uint2 u = *reinterpret_cast<const uint2*>(vp);
        a[0] = bf_lo(u.x);
        a[1] = bf_hi(u.x);
        a[2] = bf_lo(u.y);
        a[3] = bf_hi(u.y);
      } else {
        const uint32_t u = *reinterpret_cast<const uint32_t*>(vp);
        a[0] = bf_lo(u);
        a[1] = bf_hi(u);
      }
#pragma unroll
      for (int tt = 0; tt < NT; tt++) o[tt] = __builtin_amdgcn_mfma_f32_32x32x2f32(a[tt], p[v], o[tt], 0, 0, 0);
    }
    wave_lds_sync();  // the tile is rewritten next step
  }
  __syncthreads();  // every wave is done with its V tile: the area holds the waves' o now

  // the wave's (m, l, o) to LDS: o[query][dim], dims 16-row block by block
  float* ow = reinterpret_cast<float*>(lbase) + (size_t)w * 32 * DH;
  float* mlw = reinterpret_cast<float*>(lbase + LA::kMain) + (size_t)w * 64;
  if (hf == 0) {
    mlw[col] = m_run;
    mlw[32 + col] = l_run;
  }
#pragma unroll
  for (int v = 0; v < 16; v++) {
    const int i = 8 * (v >> 2) + 4 * hf + (v & 3);
    if constexpr (NT == 4) {
      *reinterpret_cast<float4*>(ow + (size_t)col * DH + i * 4) = make_float4(o[0][v], o[1][v], o[2][v], o[3][v]);
    } else {
      *reinterpret_cast<float2*>(ow + (size_t)col * DH + i * 2) = make_float2(o[0][v], o[1][v]);
    }
  }
  __syncthreads();

  // combine the waves in wave order per (query, dim pair); write a one-split row's output, else the
  // row's split record. A query of a row that has keys in this split has a valid key in wave 0's
  // first tile (key k0), so M is finite.
  constexpr int NPAIR = 32 * DH / 2, PPT = NPAIR / kWG;
  const float* mlb = reinterpret_cast<const float*>(lbase + LA::kMain);
#pragma unroll
  for (int i = 0; i < PPT; i++) {
    const int e = tid + i * kWG, j = e / (DH / 2), dp = e % (DH / 2);
    const int r = j / G, h = j % G;
    if (j >= M || k0 > pos0 + r) continue;  // no query, or no key of this split for the row
    float Mx = -INFINITY;
#pragma unroll
    for (int wv = 0; wv < LA::kWaves; wv++) Mx = fmaxf(Mx, mlb[wv * 64 + j]);
    float L = 0.f, a0 = 0.f, a1 = 0.f;
#pragma unroll
    for (int wv = 0; wv < LA::kWaves; wv++) {
      const float mw = mlb[wv * 64 + j];
      if (mw != -INFINITY) {
        const float f = expf(mw - Mx);
        L = fmaf(mlb[wv * 64 + 32 + j], f, L);
        const float2 ov = *reinterpret_cast<const float2*>(reinterpret_cast<const float*>(lbase) +
                                                           ((size_t)wv * 32 + j) * DH + 2 * dp);
        a0 = fmaf(ov.x, f, a0);
        a1 = fmaf(ov.y, f, a1);
      }
    }
    const int nsplit = (pos0 + r + C.chunk) / C.chunk;
    if (nsplit == 1) {
      const float inv = 1.0f / L;
      *reinterpret_cast<float2*>(out + (size_t)r * C.qdim + (size_t)(g * G + h) * DH + 2 * dp) =
          make_float2(a0 * inv, a1 * inv);
    } else {
      float* rec = part + ((size_t)(r * C.hkv + g) * C.max_splits + split) * RS;
      st_dev2f(rec + h * DH + 2 * dp, a0, a1);
      if (dp == 0) {
        st_dev(rec + MAXQ * DH + h, Mx);
        st_dev(rec + MAXQ * DH + MAXQ + h, L);
      }
    }
  }
  wait_own_stores();
  __syncthreads();
  if (tid < nrows) {
    const int r = tid, nsplit = (pos0 + r + C.chunk) / C.chunk;
    int last = 0;
    if (nsplit > 1 && split < nsplit) {
      const int tk = __hip_atomic_fetch_add(cnt + r * C.hkv + g, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      last = tk == nsplit - 1;
    }
    s_last[r] = last;
  }
  __syncthreads();
  float* sm = reinterpret_cast<float*>(lbase);  // the merge's (m, l) staging (the wave areas are free)
  for (int r = 0; r < nrows; r++) {
    if (!s_last[r]) continue;  // workgroup-uniform
    const int nsplit = (pos0 + r + C.chunk) / C.chunk;
    attn_merge<DH>(part + (size_t)(r * C.hkv + g) * C.max_splits * RS, nsplit, G,
                   out + (size_t)r * C.qdim + (size_t)g * G * DH, sm);
    if (tid == 0) __hip_atomic_store(cnt + r * C.hkv + g, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();  // the staging area is reused by the next row's merge
  }
}

// One split. kvb: the layer's
// cache; q: the G rotated query rows of this head group; out: their G output rows; rec_base: the
// (o[8][DH], m[8], l[8]) records of this (stage, head), one per split; cnt: its split ticket (zero at
// rest); page0: the physical page of this thread's key in the first round (key k0 + threadIdx.x / 4,
// clamped; requested by the caller before anything else). Returns true when this workgroup wrote the
// final output.
template <typename KVT, int DH>
__device__ bool attn_split(const Ctx& C, const KVT* kvb, const float* q, float* out, float* rec_base, int* cnt, int g,
                           int split, int nsplit, int k0, int k1, int pos0, int page0, float* lds) {
  if (C.G <= 4)
    return attn_split_g<KVT, DH, 4>(C, kvb, q, out, rec_base, cnt, g, split, nsplit, k0, k1, pos0, page0, lds);
  return attn_split_g<KVT, DH, 8>(C, kvb, q, out, rec_base, cnt, g, split, nsplit, k0, k1, pos0, page0, lds);
}

}  // namespace spd
