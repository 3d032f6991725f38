// Grouped fp32 GEMMs on the CDNA4 matrix cores (v_mfma_f32_32x32x2_f32).
//
// Two kernel families cover every expert contraction of the training step:
//
//  * gemm_rows: C[r, :] = op(A)[r, :] x B_g for the rows r of group g.
//    A is a slot buffer [M, K] (row r = one routed edge token, grouped by
//    expert), B_g the expert weight, stored [K, N] ("NN") or [N, K] ("NT").
//    The A loader may transform elements on the way in (SiLU of stored
//    pre-activations, ...) and the epilogue functor decides what is written
//    (plain store, gate scaling, SiLU'/SiLU'' products of the double
//    backward, per-row partial sums).
//
//  * gemm_wgrad: G_g[p, q] = sum_{r in group g} A[r, p] B[r, q], the weight
//    gradients, whose contraction runs over the tokens of an expert.  The
//    rows of each group are cut into chunks; each chunk writes a partial
//    P x Q block and a second kernel adds the chunks of a group in order,
//    so the result does not depend on scheduling.
//
// Work decomposition: a workgroup of 256 threads (4 waves as 2 x 2) owns a
// 128 x 128 output tile; each wave owns 64 x 64 = 2 x 2 MFMA blocks of
// 32 x 32, i.e. 64 accumulator floats per lane.  K advances in stages of 16
// through double-buffered LDS.  Inside a stage the k index of MFMA step s
// for lane half hf is 8g + 4hf + s (g = 0, 1), so an operand stored
// k-contiguous is read from LDS with one 16-byte load per lane per 8 k, and
// an operand stored m-contiguous with 4-byte loads whose 32-lane halves read
// consecutive words.
#pragma once

#include "common.h"

namespace janus {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int GBM = 128;            // tile rows
constexpr int GBN = 128;            // tile cols
constexpr int GBK = 16;             // k per LDS stage
constexpr int LD_MK = GBK + 4;      // row stride of an [m][k] LDS tile (floats)
constexpr int LD_KM = GBM + 8;      // row stride of a [k][m] LDS tile (floats)

struct RowsTile {   // one 128-row tile of a group
  int group;
  int r0;           // first row (global)
  int r1;           // one past the last row of the group
  int pad;
};

// ---------------------------------------------------------------- A loaders
// A loader returns 4 consecutive k-elements of row r starting at column k.

struct LoadPlain {
  const float* p;
  long long ld;
  __device__ __forceinline__ float4 operator()(long long r, int k) const {
    return *reinterpret_cast<const float4*>(p + r * ld + k);
  }
};

struct LoadSilu {   // SiLU of stored pre-activations
  const float* p;
  long long ld;
  __device__ __forceinline__ float4 operator()(long long r, int k) const {
    float4 v = *reinterpret_cast<const float4*>(p + r * ld + k);
    return make_float4(silu(v.x), silu(v.y), silu(v.z), silu(v.w));
  }
};

struct LoadRowScale {   // s[r] * p[r, k]
  const float* p;
  const float* s;
  long long ld;
  __device__ __forceinline__ float4 operator()(long long r, int k) const {
    float4 v = *reinterpret_cast<const float4*>(p + r * ld + k);
    float a = s[r];
    return make_float4(a * v.x, a * v.y, a * v.z, a * v.w);
  }
};

struct LoadSiluD1Scaled {   // SiLU'(z[r, k]) * w[k]
  const float* z;
  const float* w;
  long long ld;
  __device__ __forceinline__ float4 operator()(long long r, int k) const {
    float4 v = *reinterpret_cast<const float4*>(z + r * ld + k);
    return make_float4(silu_d1(v.x) * w[k], silu_d1(v.y) * w[k + 1], silu_d1(v.z) * w[k + 2],
                       silu_d1(v.w) * w[k + 3]);
  }
};

// ---------------------------------------------------------------- epilogues
// An epilogue sees (row, col, value) for every valid output element.

struct EpiStore {
  float* c;
  long long ld;
  static constexpr bool kRowSum = false;
  __device__ __forceinline__ float operator()(long long r, int col, float v) const {
    c[r * ld + col] = v;
    return 0.f;
  }
  __device__ __forceinline__ void rowsum(long long, int, float) const {}
};

struct EpiRowScale {   // c = s[r] * v
  float* c;
  const float* s;
  long long ld;
  static constexpr bool kRowSum = false;
  __device__ __forceinline__ float operator()(long long r, int col, float v) const {
    c[r * ld + col] = s[r] * v;
    return 0.f;
  }
  __device__ __forceinline__ void rowsum(long long, int, float) const {}
};

// ------------------------------------------------------------ LDS staging

template <class ALoad>
__device__ __forceinline__ void load_a_stage(const ALoad& al, int r0, int r1, int k0, int tid,
                                             float4 (&ra)[2]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    int q = tid + 256 * i;
    int m = q >> 2, kq = q & 3;
    long long r = (long long)r0 + m;
    ra[i] = (r < r1) ? al(r, k0 + 4 * kq) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
}

__device__ __forceinline__ void store_mk(float* s, int tid, const float4 (&ra)[2]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    int q = tid + 256 * i;
    int m = q >> 2, kq = q & 3;
    *reinterpret_cast<float4*>(s + m * LD_MK + 4 * kq) = ra[i];
  }
}

__device__ __forceinline__ void store_km(float* s, int tid, const float4 (&rb)[2]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    int q = tid + 256 * i;
    int k = q >> 5, mq = q & 31;
    *reinterpret_cast<float4*>(s + k * LD_KM + 4 * mq) = rb[i];
  }
}

// B operand of gemm_rows.  NT: B_g stored [N, K] (k-contiguous) -> [n][k] LDS.
// NN: B_g stored [K, N] (n-contiguous) -> [k][n] LDS.
template <bool NT>
__device__ __forceinline__ void load_b_stage(const float* __restrict__ Bg, int K, int N, int n0,
                                             int k0, int tid, float4 (&rb)[2]) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    int q = tid + 256 * i;
    if (NT) {
      int n = q >> 2, kq = q & 3;
      int col = n0 + n;
      rb[i] = (col < N) ? *reinterpret_cast<const float4*>(Bg + (long long)col * K + k0 + 4 * kq)
                        : make_float4(0.f, 0.f, 0.f, 0.f);
    } else {
      int k = q >> 5, nq = q & 31;
      int col = n0 + 4 * nq;
      rb[i] = (col < N) ? *reinterpret_cast<const float4*>(Bg + (long long)(k0 + k) * N + col)
                        : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  }
}

// ---------------------------------------------------------------- gemm_rows

template <bool NT, class ALoad, class Epi>
__global__ __launch_bounds__(256) void gemm_rows_kernel(ALoad al, const float* __restrict__ B,
                                                        int K, int N,
                                                        const RowsTile* __restrict__ tiles,
                                                        const int* __restrict__ n_tiles, Epi epi,
                                                        float* __restrict__ rowsum_out) {
  const int t = blockIdx.x;
  if (t >= *n_tiles) return;
  const RowsTile tile = tiles[t];
  const int n0 = blockIdx.y * GBN;
  const int r0 = tile.r0, r1 = tile.r1;
  const float* Bg = B + (long long)tile.group * K * N;

  __shared__ __attribute__((aligned(16))) float sA[2][GBM * LD_MK];
  __shared__ __attribute__((aligned(16))) float sB[2][NT ? GBN * LD_MK : GBK * LD_KM];

  const int tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63;
  const int wm = w >> 1, wn = w & 1;
  const int lr = l & 31, hf = l >> 5;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  float4 ra[2], rb[2];
  load_a_stage(al, r0, r1, 0, tid, ra);
  load_b_stage<NT>(Bg, K, N, n0, 0, tid, rb);
  store_mk(sA[0], tid, ra);
  if (NT) store_mk(sB[0], tid, rb); else store_km(sB[0], tid, rb);
  __syncthreads();

  const int nk = K / GBK;
  int cur = 0;
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) {
      load_a_stage(al, r0, r1, (kt + 1) * GBK, tid, ra);
      load_b_stage<NT>(Bg, K, N, n0, (kt + 1) * GBK, tid, rb);
    }
    const float* a_s = sA[cur];
    const float* b_s = sB[cur];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      float4 af[2];
      float bf[2][4];
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
        af[bi] = *reinterpret_cast<const float4*>(a_s + (wm * 64 + bi * 32 + lr) * LD_MK + 8 * g + 4 * hf);
#pragma unroll
      for (int bj = 0; bj < 2; ++bj) {
        if (NT) {
          float4 v = *reinterpret_cast<const float4*>(b_s + (wn * 64 + bj * 32 + lr) * LD_MK + 8 * g + 4 * hf);
          bf[bj][0] = v.x; bf[bj][1] = v.y; bf[bj][2] = v.z; bf[bj][3] = v.w;
        } else {
#pragma unroll
          for (int s = 0; s < 4; ++s) bf[bj][s] = b_s[(8 * g + 4 * hf + s) * LD_KM + wn * 64 + bj * 32 + lr];
        }
      }
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int bi = 0; bi < 2; ++bi) {
          float a = s == 0 ? af[bi].x : s == 1 ? af[bi].y : s == 2 ? af[bi].z : af[bi].w;
#pragma unroll
          for (int bj = 0; bj < 2; ++bj)
            acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, bf[bj][s], acc[bi][bj], 0, 0, 0);
        }
      }
    }
    if (more) {
      store_mk(sA[cur ^ 1], tid, ra);
      if (NT) store_mk(sB[cur ^ 1], tid, rb); else store_km(sB[cur ^ 1], tid, rb);
    }
    __syncthreads();
    cur ^= 1;
  }

  // Epilogue.  Lane l of block (bi, bj) holds column lr and rows
  // 8 (v / 4) + 4 hf + (v % 4), v = 0..15.
  float part[2][16];
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int v = 0; v < 16; ++v) part[bi][v] = 0.f;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi) {
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) {
      const int col = n0 + wn * 64 + bj * 32 + lr;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const long long row = (long long)r0 + wm * 64 + bi * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
        if (row < r1 && col < N) part[bi][v] += epi(row, col, acc[bi][bj][v]);
      }
    }
  }
  if (Epi::kRowSum) {
    // Sum over the 128 columns of the tile: 32 lanes of a half, then the two
    // column waves through LDS.  Written to rowsum_out[row * gridDim.y + blockIdx.y].
    __shared__ float red[2][GBM];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi)
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float x = part[bi][v];
#pragma unroll
        for (int o = 16; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
        part[bi][v] = x;
      }
    if (lr == 0) {
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int v = 0; v < 16; ++v) red[wn][wm * 64 + bi * 32 + 8 * (v >> 2) + 4 * hf + (v & 3)] = part[bi][v];
    }
    __syncthreads();
    if (tid < GBM) {
      const long long row = (long long)r0 + tid;
      if (row < r1) rowsum_out[row * gridDim.y + blockIdx.y] = red[0][tid] + red[1][tid];
    }
  }
}

// --------------------------------------------------------------- gemm_wgrad
// Both operands are row-major over the contraction index r: A [M, P], B [M, Q].

struct WChunk {
  int group;
  int r0;
  int r1;
  int pad;
};

template <class ALoad, class BLoad>
__global__ __launch_bounds__(256) void gemm_wgrad_kernel(ALoad al, BLoad bl, int P, int Q,
                                                         const WChunk* __restrict__ chunks,
                                                         const int* __restrict__ n_chunks,
                                                         float* __restrict__ partial) {
  const int c = blockIdx.x;
  if (c >= *n_chunks) return;
  const WChunk ch = chunks[c];
  const int ntq = (Q + GBN - 1) / GBN;
  const int p0 = (blockIdx.y / ntq) * GBM;
  const int q0 = (blockIdx.y % ntq) * GBN;

  __shared__ __attribute__((aligned(16))) float sA[2][GBK * LD_KM];
  __shared__ __attribute__((aligned(16))) float sB[2][GBK * LD_KM];

  const int tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63;
  const int wm = w >> 1, wn = w & 1;
  const int lr = l & 31, hf = l >> 5;

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

  auto load = [&](int rk, float4 (&ra)[2], float4 (&rb)[2]) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      int q = tid + 256 * i;
      int k = q >> 5, mq = q & 31;
      long long r = (long long)rk + k;
      bool rv = r < ch.r1;
      int pc = p0 + 4 * mq, qc = q0 + 4 * mq;
      ra[i] = (rv && pc < P) ? al(r, pc) : make_float4(0.f, 0.f, 0.f, 0.f);
      rb[i] = (rv && qc < Q) ? bl(r, qc) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
  };

  float4 ra[2], rb[2];
  load(ch.r0, ra, rb);
  store_km(sA[0], tid, ra);
  store_km(sB[0], tid, rb);
  __syncthreads();

  const int nk = (ch.r1 - ch.r0 + GBK - 1) / GBK;
  int cur = 0;
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    if (more) load(ch.r0 + (kt + 1) * GBK, ra, rb);
    const float* a_s = sA[cur];
    const float* b_s = sB[cur];
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      float af[2][4], bf[2][4];
#pragma unroll
      for (int s = 0; s < 4; ++s) {
#pragma unroll
        for (int bi = 0; bi < 2; ++bi) af[bi][s] = a_s[(8 * g + 4 * hf + s) * LD_KM + wm * 64 + bi * 32 + lr];
#pragma unroll
        for (int bj = 0; bj < 2; ++bj) bf[bj][s] = b_s[(8 * g + 4 * hf + s) * LD_KM + wn * 64 + bj * 32 + lr];
      }
#pragma unroll
      for (int s = 0; s < 4; ++s)
#pragma unroll
        for (int bi = 0; bi < 2; ++bi)
#pragma unroll
          for (int bj = 0; bj < 2; ++bj)
            acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[bi][s], bf[bj][s], acc[bi][bj], 0, 0, 0);
    }
    if (more) {
      store_km(sA[cur ^ 1], tid, ra);
      store_km(sB[cur ^ 1], tid, rb);
    }
    __syncthreads();
    cur ^= 1;
  }

  float* out = partial + (long long)c * P * Q;
#pragma unroll
  for (int bi = 0; bi < 2; ++bi)
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) {
      const int qc = q0 + wn * 64 + bj * 32 + lr;
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int pr = p0 + wm * 64 + bi * 32 + 8 * (v >> 2) + 4 * hf + (v & 3);
        if (pr < P && qc < Q) out[(long long)pr * Q + qc] = acc[bi][bj][v];
      }
    }
}

}  // namespace janus
