// Ragged paged decode attention as a call of its own: up to eight query rows of one layer, row i
// attending keys [0, lens[i]) of a paged KV pool (Section 3.1: each in-flight token attends, at its
// own position, over the cache of the layer it is on). It runs the step's attention split
// (attn_split_g): one workgroup per (key split, KV head, row), the split that finishes last merging
// the row's splits in split order.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>
#include <string>

#include "spd_dev.h"
#include "spd_devfn.h"
#include "spd_attn.h"

namespace spd {

void set_call_error(const std::string& msg);  // spd_last_error(NULL) (spd_api.cpp)

namespace {

struct RaggedRows {
  int lens[kMaxRows];
};

// Grid: x = key split, y = KV head, z = row. Workgroups past a row's last split return at once.
template <typename KVT, int DH, int GP>
__global__ __launch_bounds__(kWG) void k_attn_ragged(Ctx C, const float* q, const KVT* kv, float* out, float* part,
                                                     int* cnt, RaggedRows R, int smax) {
  extern __shared__ __align__(16) float lds[];
  const int split = blockIdx.x, g = blockIdx.y, z = blockIdx.z;
  const int k0 = split * C.chunk;
  const int page0 = C.page_table[min((k0 + (int)threadIdx.x / kAttnTPK) / C.page, C.max_pages - 1)];
  const int len = R.lens[z];
  const int nsplit = (len + C.chunk - 1) / C.chunk;
  if (split >= nsplit) return;
  const int k1 = min(len, k0 + C.chunk);
  constexpr int RS = kAttnMaxQ * (DH + 2);
  const size_t row = (size_t)z * C.qdim + (size_t)g * C.G * DH;
  const int cidx = z * C.hkv + g;
  attn_split_g<KVT, DH, GP>(C, kv, q + row, out + row, part + (size_t)cidx * smax * RS, cnt + cidx, g, split,
                            nsplit, k0, k1, len - 1, page0, lds);
}

__global__ __launch_bounds__(kWG) void k_zero_i32(int* p, int n) {
  for (int i = blockIdx.x * kWG + threadIdx.x; i < n; i += gridDim.x * kWG) p[i] = 0;
}

// A checked request: shapes, split count and the scratch it needs.
struct Request {
  Ctx C;
  RaggedRows R;
  int nrows, smax, dh, g4, bf16;
  size_t rec_floats;  // split records
  int tickets;        // one per (row, KV head)
};

spd_status check(const float* q, const void* kv, const int32_t* page_table, int32_t num_pages, const int32_t* lens,
                 int32_t nrows, int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim, int32_t dtype,
                 int32_t chunk, const float* out, Request* rq) {
  auto bad = [](const char* m) {
    set_call_error(m);
    return SPD_E_INVAL;
  };
  if (!q || !kv || !page_table || !lens || !out) return bad("decode attention: NULL pointer");
  if (nrows < 1 || nrows > kMaxRows) return bad("decode attention: nrows must be in [1, 8]");
  if (head_dim != 64 && head_dim != 128) return bad("decode attention: head_dim must be 64 or 128");
  if (n_kv_heads < 1 || n_q_heads < 1 || n_q_heads % n_kv_heads) return bad("decode attention: bad head counts");
  const int G = n_q_heads / n_kv_heads;
  if (G != 1 && G != 2 && G != 4 && G != 8) return bad("decode attention: n_q_heads / n_kv_heads must be 1, 2, 4 or 8");
  if (dtype != SPD_F32 && dtype != SPD_BF16) return bad("decode attention: dtype must be SPD_F32 or SPD_BF16");
  if (chunk < 16 || chunk % 16) return bad("decode attention: chunk must be a positive multiple of 16");
  if (num_pages < 1) return bad("decode attention: num_pages must be positive");
  int maxlen = 0;
  for (int i = 0; i < nrows; i++) {
    if (lens[i] < 1 || (long long)lens[i] > 16LL * num_pages)
      return bad("decode attention: every length must be in [1, 16 * num_pages]");
    maxlen = std::max(maxlen, (int)lens[i]);
  }
  const int smax = (maxlen + chunk - 1) / chunk;
  if (smax > kMaxSplits) return bad("decode attention: more than 64 key splits per row (raise chunk)");
  Request& r = *rq;
  std::memset(&r.C, 0, sizeof(Ctx));
  r.C.hq = n_q_heads;
  r.C.hkv = n_kv_heads;
  r.C.dh = head_dim;
  r.C.qdim = n_q_heads * head_dim;
  r.C.kvdim = n_kv_heads * head_dim;
  r.C.G = G;
  r.C.page = 16;
  r.C.chunk = chunk;
  r.C.max_pages = num_pages;
  r.C.max_splits = smax;
  r.C.scale = (float)(1.0 / std::sqrt((double)head_dim));
  r.C.page_table = page_table;
  std::memset(&r.R, 0, sizeof(RaggedRows));
  for (int i = 0; i < nrows; i++) r.R.lens[i] = lens[i];
  r.nrows = nrows;
  r.smax = smax;
  r.dh = head_dim;
  r.g4 = G <= 4;
  r.bf16 = dtype == SPD_BF16;
  r.rec_floats = (size_t)nrows * n_kv_heads * smax * kAttnMaxQ * (head_dim + 2);
  r.tickets = nrows * n_kv_heads;
  return SPD_OK;
}

template <typename KVT, int DH>
void launch_ragged(const Request& r, const float* q, const void* kv, float* out, float* part, int* cnt,
                   hipStream_t s) {
  const dim3 grid(r.smax, r.C.hkv, r.nrows);
  const size_t shm = attn_split_lds<KVT, DH>();
  if (r.g4)
    hipLaunchKernelGGL((k_attn_ragged<KVT, DH, 4>), grid, dim3(kWG), shm, s, r.C, q, (const KVT*)kv, out, part, cnt,
                       r.R, r.smax);
  else
    hipLaunchKernelGGL((k_attn_ragged<KVT, DH, 8>), grid, dim3(kWG), shm, s, r.C, q, (const KVT*)kv, out, part, cnt,
                       r.R, r.smax);
}

// Clears the tickets (a fill kernel, so that a captured call replays correctly), then the attention.
spd_status run(const Request& r, const float* q, const void* kv, float* out, float* part, int* cnt, void* stream) {
  hipStream_t s = (hipStream_t)stream;
  hipLaunchKernelGGL(k_zero_i32, dim3((r.tickets + kWG - 1) / kWG), dim3(kWG), 0, s, cnt, r.tickets);
  if (r.bf16) {
    if (r.dh == 128)
      launch_ragged<uint16_t, 128>(r, q, kv, out, part, cnt, s);
    else
      launch_ragged<uint16_t, 64>(r, q, kv, out, part, cnt, s);
  } else {
    if (r.dh == 128)
      launch_ragged<float, 128>(r, q, kv, out, part, cnt, s);
    else
      launch_ragged<float, 64>(r, q, kv, out, part, cnt, s);
  }
  const hipError_t e = hipGetLastError();
  if (e != hipSuccess) {
    set_call_error(std::string("decode attention launch: ") + hipGetErrorString(e));
    return SPD_E_HIP;
  }
  return SPD_OK;
}

size_t rec_bytes(const Request& r) { return (r.rec_floats * sizeof(float) + 255) / 256 * 256; }

// Scratch of spd_decode_attention_noalloc: the split records of at most kNoAllocRecords (row, KV head,
// split) triples at head_dim 128, then one ticket per (row, KV head). Each GPU the library runs on holds
// its own copy until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns for the current device (the array's name is a host-side stand-in).
constexpr int kNoAllocRecords = 2048;
constexpr size_t kNoAllocRecBytes = (size_t)kNoAllocRecords * kAttnMaxQ * (128 + 2) * sizeof(float);
constexpr size_t kNoAllocBytes = kNoAllocRecBytes + sizeof(int) * (size_t)kNoAllocRecords;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch`, looked up once per device with that device current.
spd_status scratch_of_current_device(void** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess || dev < 0 || dev >= kMaxDevices) {
    set_call_error(std::string("decode attention (no allocation): hipGetDevice: ") + hipGetErrorString(e));
    return SPD_E_HIP;
  }
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p) {
      set_call_error(std::string("decode attention (no allocation): hipGetSymbolAddress: ") + hipGetErrorString(e));
      return SPD_E_HIP;
    }
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return SPD_OK;
}

}  // namespace
}  // namespace spd

using namespace spd;

extern "C" spd_status spd_decode_attention(const float* q, const void* kv, const int32_t* page_table,
                                           int32_t num_pages, const int32_t* lens, int32_t nrows, int32_t n_q_heads,
                                           int32_t n_kv_heads, int32_t head_dim, int32_t dtype, int32_t chunk,
                                           float* out, void* workspace, size_t ws_bytes, void* stream) {
  Request r;
  spd_status st = check(q, kv, page_table, num_pages, lens, nrows, n_q_heads, n_kv_heads, head_dim, dtype, chunk, out,
                        &r);
  if (st != SPD_OK) return st;
  if (!workspace || ((uintptr_t)workspace & 255)) {
    set_call_error("decode attention: workspace must be non-NULL and 256-byte aligned");
    return SPD_E_INVAL;
  }
  const size_t need = rec_bytes(r) + sizeof(int) * (size_t)r.tickets;
  if (ws_bytes < need) {
    set_call_error("decode attention: workspace too small, " + std::to_string(need) + " bytes needed");
    return SPD_E_CAPACITY;
  }
  char* ws = (char*)workspace;
  return run(r, q, kv, out, (float*)ws, (int*)(ws + rec_bytes(r)), stream);
}

extern "C" spd_status spd_decode_attention_noalloc(const float* q, const void* kv, const int32_t* page_table,
                                                   int32_t num_pages, const int32_t* lens, int32_t nrows,
                                                   int32_t n_q_heads, int32_t n_kv_heads, int32_t head_dim,
                                                   int32_t dtype, int32_t chunk, float* out, void* stream) {
  Request r;
  spd_status st = check(q, kv, page_table, num_pages, lens, nrows, n_q_heads, n_kv_heads, head_dim, dtype, chunk, out,
                        &r);
  if (st != SPD_OK) return st;
  const size_t records = (size_t)r.nrows * r.C.hkv * r.smax;
  if (records > (size_t)kNoAllocRecords) {
    set_call_error("decode attention (no allocation): nrows * n_kv_heads * splits = " + std::to_string(records) +
                   " exceeds the " + std::to_string(kNoAllocRecords) + " split records of the static scratch");
    return SPD_E_CAPACITY;
  }
  void* base = nullptr;
  st = scratch_of_current_device(&base);
  if (st != SPD_OK) return st;
  char* ws = (char*)base;
  return run(r, q, kv, out, (float*)ws, (int*)(ws + kNoAllocRecBytes), stream);
}
