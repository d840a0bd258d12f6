// Device helpers shared by the gfx950 kernels: element types, 16-byte loads, bf16 conversion,
// wavefront reductions, the paged-KV offset, the staged-activation LDS layout and device-coherent
// accesses for data handed between workgroups of one launch.
#pragma once
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>
#include <math.h>

#include "spd_dev.h"

namespace spd {

// ------------------------------------------------------------------------------------------ types
template <typename T>
struct Elt;
template <>
struct Elt<float> {
  static constexpr int VE = 4;  // elements per 16-byte load
};
template <>
struct Elt<uint16_t> {
  static constexpr int VE = 8;
};

__device__ __forceinline__ float bf_lo(uint32_t u) { return __uint_as_float(u << 16); }
__device__ __forceinline__ float bf_hi(uint32_t u) { return __uint_as_float(u & 0xffff0000u); }

__device__ __forceinline__ uint16_t f2bf(float f) {  // round to nearest even (finite inputs)
  uint32_t u = __float_as_uint(f);
  u += 0x7fffu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

template <typename T>
__device__ __forceinline__ void unpack16(const uint4& v, float* o);
template <>
__device__ __forceinline__ void unpack16<float>(const uint4& v, float* o) {
  o[0] = __uint_as_float(v.x);
  o[1] = __uint_as_float(v.y);
  o[2] = __uint_as_float(v.z);
  o[3] = __uint_as_float(v.w);
}
template <>
__device__ __forceinline__ void unpack16<uint16_t>(const uint4& v, float* o) {
  o[0] = bf_lo(v.x);
  o[1] = bf_hi(v.x);
  o[2] = bf_lo(v.y);
  o[3] = bf_hi(v.y);
  o[4] = bf_lo(v.z);
  o[5] = bf_hi(v.z);
  o[6] = bf_lo(v.w);
  o[7] = bf_hi(v.w);
}

// 16-byte non-temporal load through the global address space, for data read once per step (weights,
// KV): the non-temporal hint streams it past the caches instead of allocating lines for it, which on
// gfx950 raises sustained HBM read bandwidth by about a sixth. (The pointers come from tables in
// memory, so the address space is stated to keep the compiler from emitting flat loads.)
typedef unsigned int v4u __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(1))) const v4u gv4u;
__device__ __forceinline__ uint4 ldg16(const void* p) {
  const v4u v = __builtin_nontemporal_load((gv4u*)(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

template <typename T>
__device__ __forceinline__ float ld1(const T* p, size_t i);
template <>
__device__ __forceinline__ float ld1<float>(const float* p, size_t i) { return p[i]; }
template <>
__device__ __forceinline__ float ld1<uint16_t>(const uint16_t* p, size_t i) {
  return __uint_as_float(((uint32_t)p[i]) << 16);
}

// Two consecutive elements (4- or 8-byte aligned) as floats.
template <typename T>
__device__ __forceinline__ float2 ld2(const T* p);
template <>
__device__ __forceinline__ float2 ld2<float>(const float* p) { return *reinterpret_cast<const float2*>(p); }
template <>
__device__ __forceinline__ float2 ld2<uint16_t>(const uint16_t* p) {
  const uint32_t u = *reinterpret_cast<const uint32_t*>(p);
  return make_float2(bf_lo(u), bf_hi(u));
}

template <typename T>
__device__ __forceinline__ void st1(T* p, size_t i, float v);
template <>
__device__ __forceinline__ void st1<float>(float* p, size_t i, float v) { p[i] = v; }
template <>
__device__ __forceinline__ void st1<uint16_t>(uint16_t* p, size_t i, float v) { p[i] = f2bf(v); }

// ------------------------------------------------------------------------------------ reductions
__device__ __forceinline__ float wave_sum(float v) {
  // xor butterfly: every lane ends with the same, order-fixed total (fp add is commutative)
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
  return v;
}


__device__ __forceinline__ size_t kv_off(const Ctx& C, int pos, int kvh, int j) {
  // [page][2][Hkv][page_size][dh]; returns the K element offset (V is + Hkv*page*dh)
  const int pg = C.page_table[pos / C.page];
  return (size_t)pg * (2 * C.hkv * C.page * C.dh) + ((size_t)kvh * C.page + (pos % C.page)) * C.dh + j;
}

// LDS layout of one staged activation chunk. For bf16 weights lane l multiplies columns
// 8l..8l+7 of each 512-column block; the chunk is stored so that the lane's first four and last
// four values are two conflict-free 16-byte LDS reads.
template <int VE>
__device__ __forceinline__ int xidx(int k) {
  if constexpr (VE == 8) {
    const int blk = k >> 9, w = k & 511, l = w >> 3, e = w & 7;
    return (blk << 9) + ((e >> 2) << 8) + (l << 2) + (e & 3);
  } else {
    return k;
  }
}

// Weight blocks loaded at once per row: a wave keeps RL rows x kU blocks of 16-byte loads in flight.
constexpr int kU = 5;

__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int w = threadIdx.x >> 6;
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  return (red[0] + red[1]) + (red[2] + red[3]);
}

__device__ __forceinline__ bool better(float v, int i, float bv, int bi) {
  return v > bv || (v == bv && i < bi);
}

// 64-bit argmax key: the high word orders logits (a monotone map of the float bits; NaN ranks below
// every number), the low word orders indices ascending, so the maximum key is the largest logit with
// the lowest index among equals. Zero is below every key produced here.
__device__ __forceinline__ unsigned long long argmax_key(float v, int i) {
  uint32_t u = __float_as_uint(v);
  u = (u & 0x80000000u) ? ~u : (u | 0x80000000u);
  if (v != v) u = 0u;
  return ((unsigned long long)u << 32) | (unsigned long long)(0xffffffffu - (uint32_t)i);
}
__device__ __forceinline__ int argmax_index(unsigned long long key, int V) {
  const uint32_t i = 0xffffffffu - (uint32_t)(key & 0xffffffffull);
  return i < (uint32_t)V ? (int)i : 0;  // an all-NaN row cannot produce an out-of-range id
}

// Device-coherent scalar accesses for data handed between workgroups of one launch: agent-scope
// atomic stores and loads are issued with device scope (written through to, and read from, the
// level every XCD shares), so no L2 writeback fence is needed; a producer waits for its own
// stores (s_waitcnt) before it signals.
__device__ __forceinline__ void st_dev(float* p, float v) {
  __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ float ld_dev(const float* p) {
  return __hip_atomic_load(const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void wait_own_stores() {
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
  __builtin_amdgcn_s_waitcnt(0);
  __atomic_signal_fence(__ATOMIC_SEQ_CST);
}

__device__ __forceinline__ int ld_dev_i(const int* p) {
  return __hip_atomic_load(const_cast<int*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Launch trace (debugging and measurement): slot (j * 5 + k) * n + s is sublayer k of layer slot j
// of stage s; then the LM head, verify and the PDM's feature projection. The launch's first
// workgroup (dispatched first) stores the start; every workgroup folds its end time into the slot
// with a maximum that nothing waits for, so the trace barely moves the schedule it measures.
enum KTraceExtra { KT_HEAD = 0, KT_VERIFY = 1, KT_PDM = 2, KT_EXTRA = 4 };
__device__ __forceinline__ int ktrace_slot(const Ctx& C, int j, int k, int s) { return (j * 5 + k) * C.n + s; }
__device__ __forceinline__ int ktrace_extra(const Ctx& C, int e) { return 5 * C.J * C.n + e; }
__device__ __forceinline__ void ktrace_start(const Ctx& C, int slot, bool first) {
  if (C.ktrace != nullptr && first && threadIdx.x == 0) C.ktrace[2 * slot] = (unsigned long long)wall_clock64();
}
__device__ __forceinline__ void ktrace_end(const Ctx& C, int slot) {
  if (C.ktrace != nullptr && threadIdx.x == 0)
    __hip_atomic_fetch_max(C.ktrace + 2 * slot + 1, (unsigned long long)wall_clock64(), __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
}

__device__ __forceinline__ float2 ld_dev2(const float* p) {  // p 8-byte aligned
  const unsigned long long u =
      __hip_atomic_load((unsigned long long*)const_cast<float*>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
  return make_float2(__uint_as_float((uint32_t)u), __uint_as_float((uint32_t)(u >> 32)));
}

// Host: launch on stream s, handing the timing events set by set_launch_events (if any) to the dispatch.
void current_launch_events(hipEvent_t* start, hipEvent_t* stop);
template <typename F, typename... Args>
static inline void launch_timed(F kernel, dim3 grid, dim3 block, size_t shmem, hipStream_t s, Args... args) {
  hipEvent_t a = nullptr, b = nullptr;
  current_launch_events(&a, &b);
  if (a != nullptr)
    hipExtLaunchKernelGGL(kernel, grid, block, (std::uint32_t)shmem, s, a, b, 0u, args...);
  else
    hipLaunchKernelGGL(kernel, grid, block, shmem, s, args...);
}

}  // namespace spd
