// Tables, chunk reduction and the standalone grouped-GEMM entry points.
#include <cstring>
#include <mutex>

#include "internal.h"

namespace janus {

__global__ void build_rows_tiles_kernel(const int* __restrict__ row_off, int n_groups, RowsTile* tiles,
                                        int* n_tiles) {
  __shared__ int pre[1025];
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int g = 0; g < n_groups; ++g) {
      pre[g] = acc;
      int m = row_off[g + 1] - row_off[g];
      acc += (m + GBM - 1) / GBM;
    }
    pre[n_groups] = acc;
    *n_tiles = acc;
  }
  __syncthreads();
  const int total = pre[n_groups];
  for (int t = threadIdx.x; t < total; t += blockDim.x) {
    int lo = 0, hi = n_groups;   // pre[lo] <= t < pre[hi]
    while (hi - lo > 1) {
      int mid = (lo + hi) >> 1;
      if (pre[mid] <= t) lo = mid; else hi = mid;
    }
    RowsTile e;
    e.group = lo;
    e.r0 = row_off[lo] + (t - pre[lo]) * GBM;
    e.r1 = row_off[lo + 1];
    e.pad = 0;
    tiles[t] = e;
  }
}

__global__ void build_wchunks_kernel(const int* __restrict__ row_off, int n_groups, int kc, WChunk* chunks,
                                     int* n_chunks, int* chunk_first) {
  __shared__ int pre[1025];
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int g = 0; g < n_groups; ++g) {
      pre[g] = acc;
      chunk_first[g] = acc;
      int m = row_off[g + 1] - row_off[g];
      acc += (m + kc - 1) / kc;
    }
    pre[n_groups] = acc;
    chunk_first[n_groups] = acc;
    *n_chunks = acc;
  }
  __syncthreads();
  const int total = pre[n_groups];
  for (int t = threadIdx.x; t < total; t += blockDim.x) {
    int lo = 0, hi = n_groups;
    while (hi - lo > 1) {
      int mid = (lo + hi) >> 1;
      if (pre[mid] <= t) lo = mid; else hi = mid;
    }
    WChunk e;
    e.group = lo;
    e.r0 = row_off[lo] + (t - pre[lo]) * kc;
    e.r1 = min(e.r0 + kc, row_off[lo + 1]);
    e.pad = 0;
    chunks[t] = e;
  }
}

// G_g (+)= sum of the chunk partials of group g.  A workgroup owns 16
// float4 columns; its 16 column-slices sum the chunks c0 + s, c0 + s + 16, ...
// (two accumulators each), and the slices are added in order 0..15, so the
// result is the same on every run.
constexpr int kRedSlices = 16;
__global__ void wgrad_reduce_kernel(const float* __restrict__ partial, const int* __restrict__ chunk_first,
                                    int n_groups, long long PQ, float* __restrict__ G, int accumulate) {
  __shared__ float4 red[kRedSlices][16];
  const int g = blockIdx.y;
  const int cl = threadIdx.x & 15, sl = threadIdx.x >> 4;
  const long long i4 = (long long)blockIdx.x * 16 + cl;
  const bool ok = 4 * i4 < PQ;
  const int c0 = chunk_first[g], c1 = chunk_first[g + 1];
  float4 a = make_float4(0.f, 0.f, 0.f, 0.f), b = a;
  if (ok) {
    int c = c0 + sl;
    for (; c + kRedSlices < c1; c += 2 * kRedSlices) {
      const float4 u = reinterpret_cast<const float4*>(partial + (long long)c * PQ)[i4];
      const float4 v = reinterpret_cast<const float4*>(partial + (long long)(c + kRedSlices) * PQ)[i4];
      a.x += u.x; a.y += u.y; a.z += u.z; a.w += u.w;
      b.x += v.x; b.y += v.y; b.z += v.z; b.w += v.w;
    }
    if (c < c1) {
      const float4 u = reinterpret_cast<const float4*>(partial + (long long)c * PQ)[i4];
      a.x += u.x; a.y += u.y; a.z += u.z; a.w += u.w;
    }
  }
  red[sl][cl] = make_float4(a.x + b.x, a.y + b.y, a.z + b.z, a.w + b.w);
  __syncthreads();
  if (sl == 0 && ok) {
    float4* out = reinterpret_cast<float4*>(G + (long long)g * PQ) + i4;
    float4 s = accumulate ? *out : make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
    for (int q = 0; q < kRedSlices; ++q) {
      const float4 v = red[q][cl];
      s.x += v.x; s.y += v.y; s.z += v.z; s.w += v.w;
    }
    *out = s;
  }
}

int skinny_chunk_rows(long long M, int P, int Q) {
  const size_t lds = sizeof(float) * P * Q;
  int per_cu = 0, dev = 0, cus = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
  if (e == hipSuccess) e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, skinny_kernel(P, Q), 256, lds);
  const long long slots = (e == hipSuccess && per_cu > 0 && cus > 0) ? (long long)per_cu * cus : 1024;
  const long long R = skinny_rows(Q);
  const long long per = (M + slots - 1) / slots;
  const long long kc = ((per + R - 1) / R) * R;
  return (int)(kc < R ? R : kc);
}

void launch_wgrad_reduce(hipStream_t st, const float* partial, const int* chunk_first, int groups,
                         long long PQ, float* G, int accumulate) {
  dim3 rg(cdiv(PQ / 4, 16), groups);
  hipLaunchKernelGGL(wgrad_reduce_kernel, rg, dim3(16 * kRedSlices), 0, st, partial, chunk_first, groups, PQ, G,
                     accumulate);
}

// Tile and chunk tables from group row offsets (one workgroup).
void build_tables(hipStream_t st, const int* row_off, int groups, int kc, RowsTile* tiles, int* n_tiles,
                  WChunk* chunks, int* n_chunks, int* chunk_first) {
  if (tiles) hipLaunchKernelGGL(build_rows_tiles_kernel, dim3(1), dim3(256), 0, st, row_off, groups, tiles, n_tiles);
  if (chunks)
    hipLaunchKernelGGL(build_wchunks_kernel, dim3(1), dim3(256), 0, st, row_off, groups, kc, chunks, n_chunks,
                       chunk_first);
}

int ensure(janus_buffer& b, size_t bytes) {
  if (bytes <= b.bytes && b.ptr) return JANUS_OK;
  if (b.ptr) {
    hipError_t e = hipFree(b.ptr);
    b.ptr = nullptr;
    b.bytes = 0;
    if (e != hipSuccess) return janus_set_hip_error(e);
  }
  size_t want = bytes < 256 ? 256 : bytes;
  if (hipMalloc(&b.ptr, want) != hipSuccess) {
    (void)hipGetLastError();
    b.ptr = nullptr;
    return JANUS_ENOMEM;
  }
  b.bytes = want;
  return JANUS_OK;
}

}  // namespace janus

using namespace janus;

extern "C" int janus_grouped_gemm(janus_ctx* ctx, const float* A, const float* B, float* C,
                                  const int32_t* row_off, int32_t n_groups, int64_t M, int32_t K, int32_t N,
                                  int32_t trans_b, void* stream) {
  if (!ctx || (M > 0 && (!A || !C)) || !B || !row_off || n_groups < 1 || n_groups > 1024 || M < 0 || M > INT32_MAX ||
      K <= 0 || K % GBK || N <= 0 || N % 64)
    return JANUS_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int mt = max_rows_tiles(M, n_groups);
  Carver cv(nullptr);
  cv.take<RowsTile>(mt);
  cv.take<int>(1);
  int rc = ensure(ctx->aux, cv.size());
  if (rc) return rc;
  Carver c2(ctx->aux.ptr);
  RowsTile* tiles = c2.take<RowsTile>(mt);
  int* nt = c2.take<int>(1);
  build_tables(st, row_off, n_groups, 0, tiles, nt, nullptr, nullptr, nullptr);
  if (trans_b)
    launch_rows<true>(st, LoadPlain{A, K}, B, K, N, tiles, nt, mt, EpiStore{C, N});
  else
    launch_rows<false>(st, LoadPlain{A, K}, B, K, N, tiles, nt, mt, EpiStore{C, N});
  JANUS_HIP_TRY(hipGetLastError());
  return JANUS_OK;
}

// Fixed scratch of janus_grouped_gemm_noalloc: the tile table and its count.
// One copy per device, allocated with the library's code object on that
// device and held until the process ends; host code uses only the address
// returned by hipGetSymbolAddress for the current device, never the symbol.
constexpr size_t kNoAllocScratchBytes = size_t(4) << 20;
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

namespace {

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxDevices] = {};

// Address of the current device's scratch, looked up once per device.
int noalloc_scratch(void** out) {
  int dev = 0;
  JANUS_HIP_TRY(hipGetDevice(&dev));
  if (dev < 0 || dev >= kMaxDevices) return JANUS_EUNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    JANUS_HIP_TRY(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) return JANUS_EHIP;
    g_scratch_ptr[dev] = p;
  }
  *out = g_scratch_ptr[dev];
  return JANUS_OK;
}

}  // namespace

// Largest tile table the fixed scratch holds (tiles first, then the count).
static int noalloc_max_tiles() {
  return (int)((kNoAllocScratchBytes - 256) / sizeof(RowsTile));
}

extern "C" int janus_grouped_gemm_noalloc(const float* A, const float* B, float* C, const int32_t* row_off,
                                          int32_t n_groups, int64_t M, int32_t K, int32_t N, int32_t trans_b,
                                          void* stream) {
  if ((M > 0 && (!A || !C)) || !B || !row_off || n_groups < 1 || n_groups > 1024 || M < 0 || M > INT32_MAX ||
      K <= 0 || K % GBK || N <= 0 || N % 64)
    return JANUS_EINVAL;
  const int mt = max_rows_tiles(M, n_groups);
  if (mt > noalloc_max_tiles()) return JANUS_ENOMEM;
  void* base = nullptr;
  int rc = noalloc_scratch(&base);
  if (rc) return rc;
  hipStream_t st = static_cast<hipStream_t>(stream);
  Carver cv(base);
  RowsTile* tiles = cv.take<RowsTile>(mt);
  int* nt = cv.take<int>(1);
  if (cv.size() > kNoAllocScratchBytes) return JANUS_ENOMEM;
  // the table kernel rewrites the count and every tile the launch reads, so
  // nothing left by an earlier call is used
  build_tables(st, row_off, n_groups, 0, tiles, nt, nullptr, nullptr, nullptr);
  if (trans_b)
    launch_rows<true>(st, LoadPlain{A, K}, B, K, N, tiles, nt, mt, EpiStore{C, N});
  else
    launch_rows<false>(st, LoadPlain{A, K}, B, K, N, tiles, nt, mt, EpiStore{C, N});
  JANUS_HIP_TRY(hipGetLastError());
  return JANUS_OK;
}

extern "C" int32_t janus_wgrad_chunk_rows(int64_t M, int32_t P, int32_t Q) {
  if (M < 0 || M > INT32_MAX || P <= 0 || Q <= 0) return JANUS_EINVAL;
  return wgrad_chunk_rows(M, P, Q);
}

extern "C" int janus_grouped_wgrad(janus_ctx* ctx, const float* A, const float* B, float* G,
                                   const int32_t* row_off, int32_t n_groups, int64_t M, int32_t P, int32_t Q,
                                   void* stream) {
  if (!ctx || (M > 0 && (!A || !B)) || !G || !row_off || n_groups < 1 || n_groups > 1024 || M < 0 || M > INT32_MAX ||
      P <= 0 || P % 4 || Q <= 0 || Q % 4)
    return JANUS_EINVAL;
  hipStream_t st = static_cast<hipStream_t>(stream);
  const int kc = wgrad_chunk_rows(M, P, Q);
  const int mc = max_wchunks(M, n_groups, kc);
  Carver cv(nullptr);
  cv.take<WChunk>(mc);
  cv.take<int>(1);
  cv.take<int>(n_groups + 1);
  cv.take<float>((size_t)mc * P * Q);
  int rc = ensure(ctx->aux, cv.size());
  if (rc) return rc;
  Carver c2(ctx->aux.ptr);
  WChunk* chunks = c2.take<WChunk>(mc);
  int* nc = c2.take<int>(1);
  int* first = c2.take<int>(n_groups + 1);
  float* partial = c2.take<float>((size_t)mc * P * Q);
  build_tables(st, row_off, n_groups, kc, nullptr, nullptr, chunks, nc, first);
  launch_wgrad(st, LoadPlain{A, P}, LoadPlain{B, Q}, P, Q, chunks, nc, first, mc, n_groups, partial, G, 0);
  JANUS_HIP_TRY(hipGetLastError());
  return JANUS_OK;
}
