// Grouped fp32 GEMMs on the CDNA4 matrix cores (v_mfma_f32_32x32x2_f32).
//
// Two kernel families cover every expert contraction of the training step:
//
//  * gemm_rows: C[r, :] = op(A)[r, :] x B_g for the rows r of group g.
//    A is a slot buffer [M, K] (row r = one routed edge token, grouped by
//    expert), B_g the expert weight, stored [K, N] ("NN") or [N, K] ("NT").
//    The A loader may transform elements on their way into LDS (SiLU of
//    stored pre-activations, ...) and the epilogue functor decides what is
//    written (plain store, gate scaling, the SiLU'/SiLU'' products of the
//    double backward, per-row partial sums).
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
// through double-buffered LDS; the global loads of stage s+1 are in flight
// while stage s is multiplied.  Operands stored as they are used (the expert
// weights, and every slot-row operand without a transform) go from global
// memory straight into LDS (global_load_lds_dwordx4: no registers, no LDS
// store instructions); an operand transform (SiLU of stored pre-activations,
// a row scale) runs when its registers are written to LDS, and so do the
// zeros of a weight-gradient chunk's last partial stage.  Inside a stage the
// k index of MFMA step j for lane half hf is 8g + 4hf + j (g = 0, 1), so an operand stored
// k-contiguous is read from LDS with one 16-byte load per lane per 8 k, and
// an operand stored m-contiguous with 4-byte loads whose 32-lane halves read
// consecutive words.
//
// Epilogue: the accumulators are staged through LDS, 64 rows at a time, and
// then visited row-major as float4, so every epilogue read and write of
// global memory is a coalesced 512-byte row segment; a thread issues the
// epilogue reads of four pieces before it uses any of them.
#pragma once

#include <type_traits>

#include "common.h"

namespace janus {

typedef float f32x16 __attribute__((ext_vector_type(16)));

constexpr int GBM = 128;            // tile rows
constexpr int GBN = 128;            // tile cols
constexpr int GBK = 16;             // k per LDS stage
constexpr int LD_MK = GBK;          // row stride of an [m][k] LDS tile (floats; float4 columns swizzled)
constexpr int LD_KM = GBM + 8;      // row stride of a [k][m] LDS tile (floats)
constexpr int LD_C = GBN + 8;       // row stride of the staged output (floats)
constexpr int cmax(int a, int b) { return a > b ? a : b; }
constexpr int B_BUF = cmax(GBN * LD_MK, GBK * LD_KM);             // one B stage, [n][k] or [k][n]
constexpr int SMEM_MAIN = cmax(2 * GBM * LD_MK + 2 * B_BUF,       // gemm_rows
                               4 * GBK * LD_KM);                   // gemm_wgrad
constexpr int SMEM_EPI = 64 * LD_C;
constexpr int SMEM_FLOATS = SMEM_MAIN > SMEM_EPI ? SMEM_MAIN : SMEM_EPI;

struct RowsTile {   // one 128-row tile of a group
  int group;
  int r0;           // first row (global)
  int r1;           // one past the last row of the group
  int pad;
};

__device__ __forceinline__ float4 f4zero() { return make_float4(0.f, 0.f, 0.f, 0.f); }
__device__ __forceinline__ float4 ld4(const float* p) { return *reinterpret_cast<const float4*>(p); }
__device__ __forceinline__ void st4(float* p, float4 v) { *reinterpret_cast<float4*>(p) = v; }
typedef float f32x4v __attribute__((ext_vector_type(4)));
// Streaming accesses of the epilogues (each element is read or written once per launch).
__device__ __forceinline__ float4 ld4nt(const float* p) {
  const f32x4v v = __builtin_nontemporal_load(reinterpret_cast<const f32x4v*>(p));
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void st4nt(float* p, float4 v) {
  const f32x4v x = {v.x, v.y, v.z, v.w};
  __builtin_nontemporal_store(x, reinterpret_cast<f32x4v*>(p));
}

// XCD-aware block order.  Workgroups are handed to the 8 XCDs round-robin
// by linear id, and each XCD has its own L2.  Block b runs on XCD b % 8 as
// that XCD's (b / 8)-th block, so the ntile output tiles that share one row
// range (or one weight-gradient chunk) are given to consecutive blocks of
// one XCD: row range r = (slot / ntile) * 8 + xcd, tile = slot % ntile.
// The grid is rows8(nrange) * ntile blocks; ids past the last range exit.
__device__ __forceinline__ void xcd_map(int b, int ntile, int& range, int& tile) {
  const int xcd = b & 7, slot = b >> 3;
  tile = slot % ntile;
  range = (slot / ntile) * 8 + xcd;
}
inline unsigned xcd_grid(long long nrange, int ntile) { return (unsigned)(((nrange + 7) / 8) * 8 * ntile); }

// ---------------------------------------------------------------- loaders
// load(r, k) fetches what element (r, k..k+3) needs from global memory;
// apply(raw, k) turns it into the 4 operand values (only for valid rows).

struct LoadPlain {
  const float* p;
  long long ld;
  using Raw = float4;
  __device__ __forceinline__ Raw load(long long r, int k) const { return ld4(p + r * ld + k); }
  __device__ __forceinline__ float4 apply(const Raw& v, int) const { return v; }
};

struct LoadSilu {   // SiLU of stored pre-activations
  const float* p;
  long long ld;
  using Raw = float4;
  __device__ __forceinline__ Raw load(long long r, int k) const { return ld4(p + r * ld + k); }
  __device__ __forceinline__ float4 apply(const Raw& v, int) const {
    return make_float4(silu(v.x), silu(v.y), silu(v.z), silu(v.w));
  }
};

struct LoadSiluRowScale {   // s[r] * SiLU(p[r, k])
  const float* p;
  const float* s;
  long long ld;
  struct Raw {
    float4 v;
    float s;
  };
  __device__ __forceinline__ Raw load(long long r, int k) const { return Raw{ld4(p + r * ld + k), s[r]}; }
  __device__ __forceinline__ float4 apply(const Raw& x, int) const {
    return make_float4(x.s * silu(x.v.x), x.s * silu(x.v.y), x.s * silu(x.v.z), x.s * silu(x.v.w));
  }
};

struct LoadSiluD1Scaled {   // SiLU'(z[r, k]) * w[k]
  const float* z;
  const float* w;
  long long ld;
  using Raw = float4;
  __device__ __forceinline__ Raw load(long long r, int k) const { return ld4(z + r * ld + k); }
  __device__ __forceinline__ float4 apply(const Raw& v, int k) const {
    const float4 ww = ld4(w + k);
    return make_float4(silu_d1(v.x) * ww.x, silu_d1(v.y) * ww.y, silu_d1(v.z) * ww.z, silu_d1(v.w) * ww.w);
  }
};

// ---------------------------------------------------------------- epilogues
// An epilogue works on output row r, columns c..c+3 (c % 4 == 0) in two
// steps so that all of a thread's global reads are in flight together:
// load(r, c) fetches what the piece needs, store(r, c, v, raw) writes the
// results and returns the piece's contribution to the row sum (kRowSum).

struct NoRaw {};

struct EpiStore {
  float* c;
  long long ld;
  static constexpr bool kRowSum = false;
  using Raw = NoRaw;
  __device__ __forceinline__ Raw load(long long, int) const { return Raw{}; }
  __device__ __forceinline__ float store(long long r, int col, float4 v, const Raw&) const {
    st4nt(c + r * ld + col, v);
    return 0.f;
  }
};

// Same store for the dense readout products (a distinct type keeps their
// kernels apart from the expert ones in profiles).
struct EpiDense : EpiStore {};

struct EpiRowScale {   // c = s[r] * v
  float* c;
  const float* s;
  long long ld;
  static constexpr bool kRowSum = false;
  using Raw = float;
  __device__ __forceinline__ Raw load(long long r, int) const { return s[r]; }
  __device__ __forceinline__ float store(long long r, int col, float4 v, const Raw& a) const {
    st4nt(c + r * ld + col, make_float4(a * v.x, a * v.y, a * v.z, a * v.w));
    return 0.f;
  }
};

// C = A B + R (residual R may be null): the attention output added to the atom features.
struct EpiAdd {
  float* c;
  const float* r;
  long long ld;
  static constexpr bool kRowSum = false;
  using Raw = float4;
  __device__ __forceinline__ Raw load(long long row, int col) const {
    return r ? ld4nt(r + row * ld + col) : make_float4(0.f, 0.f, 0.f, 0.f);
  }
  __device__ __forceinline__ float store(long long row, int col, float4 v, const Raw& x) const {
    st4nt(c + row * ld + col, make_float4(v.x + x.x, v.y + x.y, v.z + x.z, v.w + x.w));
    return 0.f;
  }
};

// Force backward, after Sbar = Ybar W2^T: keep Sbar and Abar = SiLU'(A) Sbar.
struct EpiP2 {
  const float* A;
  float* Sb;
  float* Ab;
  long long ld;
  static constexpr bool kRowSum = false;
  using Raw = float4;
  __device__ __forceinline__ Raw load(long long r, int c) const { return ld4nt(A + r * ld + c); }
  __device__ __forceinline__ float store(long long r, int c, float4 v, const Raw& a) const {
    const long long i = r * ld + c;
    st4nt(Sb + i, v);
    st4nt(Ab + i, make_float4(silu_d1(a.x) * v.x, silu_d1(a.y) * v.y, silu_d1(a.z) * v.z, silu_d1(a.w) * v.w));
    return 0.f;
  }
};

struct Float4x2 {
  float4 a, b;
};

// Double backward, after Abt = Xbt W1:
//   Sbt = SiLU'(A) Abt        (overwrites Abar, which the weight gradient has consumed)
//   C   = SiLU''(A) Sbar Abt  (overwrites Sbar; consumed by the final backward)
struct EpiP3 {
  const float* A;
  float* Sb;
  float* Ab;
  long long ld;
  static constexpr bool kRowSum = false;
  using Raw = Float4x2;
  __device__ __forceinline__ static void d12(float a, float& d1, float& d2) {
    const float s = sig(a);
    d1 = s + a * s * (1.f - s);
    d2 = s * (1.f - s) * (2.f + a * (1.f - 2.f * s));
  }
  __device__ __forceinline__ Raw load(long long r, int c) const {
    const long long i = r * ld + c;
    return Raw{ld4nt(A + i), ld4nt(Sb + i)};
  }
  __device__ __forceinline__ float store(long long r, int c, float4 v, const Raw& x) const {
    const long long i = r * ld + c;
    const float4 a = x.a, sb = x.b;
    float4 o1, o2;
    float d1, d2;
    d12(a.x, d1, d2); o1.x = d1 * v.x; o2.x = d2 * sb.x * v.x;
    d12(a.y, d1, d2); o1.y = d1 * v.y; o2.y = d2 * sb.y * v.y;
    d12(a.z, d1, d2); o1.z = d1 * v.z; o2.z = d2 * sb.z * v.z;
    d12(a.w, d1, d2); o1.w = d1 * v.w; o2.w = d2 * sb.w * v.w;
    st4nt(Ab + i, o1);
    st4nt(Sb + i, o2);
    return 0.f;
  }
};

// Final backward, after St = mt W2^T (ungated adjoint of the message):
//   At = g SiLU'(A) St + C  (overwrites C); returns St . SiLU(A) for the gate adjoint.
struct EpiP4 {
  const float* A;
  float* Sb;
  const float* gate;
  long long ld;
  static constexpr bool kRowSum = true;
  struct Raw {
    float4 a, c;
    float g;
  };
  __device__ __forceinline__ static float one(float a, float v, float c, float g, float& sum) {
    const float s = sig(a);
    sum += v * a * s;
    return g * (s + a * s * (1.f - s)) * v + c;
  }
  __device__ __forceinline__ Raw load(long long r, int c) const {
    const long long i = r * ld + c;
    return Raw{ld4nt(A + i), ld4nt(Sb + i), gate[r]};
  }
  __device__ __forceinline__ float store(long long r, int c, float4 v, const Raw& x) const {
    float sum = 0.f;
    float4 o;
    o.x = one(x.a.x, v.x, x.c.x, x.g, sum);
    o.y = one(x.a.y, v.y, x.c.y, x.g, sum);
    o.z = one(x.a.z, v.z, x.c.z, x.g, sum);
    o.w = one(x.a.w, v.w, x.c.w, x.g, sum);
    st4nt(Sb + r * ld + c, o);
    return sum;
  }
};

// ------------------------------------------------------------ LDS staging
// [m][k] tiles hold the 4 float4 columns of row m in the order
// kq ^ ((m / 4) % 4): a 16-lane group then touches 64 distinct banks both
// when it stores 4 rows x 4 columns and when it reads one column of 16 rows.
static_assert(GBK == 16, "the [m][k] swizzle assumes 4 float4 columns per row");
__device__ __forceinline__ int mk_off(int m, int kq) { return m * LD_MK + 4 * (kq ^ ((m >> 2) & 3)); }

// The loads are unconditional: rows (and columns) past the end of the range
// read the last valid one and are replaced by zeros when stored to LDS.  A
// conditional load would put a branch around every load, and at the join
// the compiler waits for all earlier loads, which serialises them.  Ranges
// are never empty (tiles and chunks are built only over rows that exist;
// widths are multiples of 4).

// [m][k] tile from a k-contiguous operand: thread q loads row q/4, k-quad q%4.
template <class L>
struct StageMK {
  typename L::Raw raw[2];
  bool ok[2];
  __device__ __forceinline__ void load(const L& ld, int r0, int r1, int k0, int tid) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      const long long r = (long long)r0 + (q >> 2);
      ok[i] = r < r1;
      raw[i] = ld.load(ok[i] ? r : (long long)r1 - 1, k0 + 4 * (q & 3));
    }
  }
  __device__ __forceinline__ void store(const L& ld, float* s, int k0, int tid) const {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      st4(s + mk_off(q >> 2, q & 3), ok[i] ? ld.apply(raw[i], k0 + 4 * (q & 3)) : f4zero());
    }
  }
};

// [k][m] tile from an m-contiguous operand: thread q loads k-row q/32, m-quad q%32.
template <class L>
struct StageKM {
  typename L::Raw raw[2];
  bool ok[2];
  __device__ __forceinline__ void load(const L& ld, long long rk, long long rk_end, int m0, int m_end, int tid) {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      const long long r = rk + (q >> 5);
      const int m = m0 + 4 * (q & 31);
      ok[i] = r < rk_end && m < m_end;
      raw[i] = ld.load(r < rk_end ? r : rk_end - 1, m < m_end ? m : m_end - 4);
    }
  }
  __device__ __forceinline__ void store(const L& ld, float* s, int m0, int tid) const {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i;
      st4(s + (q >> 5) * LD_KM + 4 * (q & 31), ok[i] ? ld.apply(raw[i], m0 + 4 * (q & 31)) : f4zero());
    }
  }
  // the same into the unpadded swizzled layout of direct_km
  __device__ __forceinline__ void store_sw(const L& ld, float* s, int m0, int tid) const {
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int q = tid + 256 * i, k = q >> 5;
      st4(s + k * GBM + ((4 * (q & 31)) ^ (((k >> 2) & 1) << 5)),
          ok[i] ? ld.apply(raw[i], m0 + 4 * (q & 31)) : f4zero());
    }
  }
};

// Direct global-to-LDS loads of one [m][k] stage of a plain operand (128 rows x 16 k):
// lane l of wave w writes the 16 bytes at LDS float (i*256 + w*64 + l)*4, which is row
// m = i*64 + w*16 + l/4, column slot l%4 of the swizzled layout, so it loads k-quad
// (l%4) ^ ((m/4)%4) of row m.  Rows past r1 load row r1 - 1 (their products are never stored).
template <class L>
struct IsPlainLoad : std::false_type {};
template <>
struct IsPlainLoad<LoadPlain> : std::true_type {};
typedef __attribute__((address_space(3))) void* lds_ptr;
__device__ __forceinline__ void direct_mk(const float* __restrict__ p, long long ld, int r0, int r1, int k0,
                                          float* s, int tid) {
  const int l = tid & 63, w = tid >> 6;
  const int kq = (l & 3) ^ ((l >> 4) & 3);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const long long r = (long long)r0 + i * 64 + w * 16 + (l >> 2);
    const float* src = p + (r < r1 ? r : (long long)r1 - 1) * ld + k0 + 4 * kq;
    __builtin_amdgcn_global_load_lds(src, (lds_ptr)(s + (i * 256 + w * 64) * 4), 16, 0, 0);
  }
}
// Direct loads of one [k][m] stage (16 k-rows x 128 columns of an m-contiguous plain
// operand) into an unpadded layout whose rows k with (k / 4) odd hold their two 32-column
// halves of each 64 swapped (column c at c ^ 32): the two half-waves of an MFMA operand
// read, rows 4 apart, then fall on different banks.  Lane l of wave w writes LDS float
// (i*256 + w*64 + l)*4: row k = i*8 + w*2 + l/32, position 4 (l % 32).  Columns past
// m_end load column m_end - 4 (their products are never stored).
__device__ __forceinline__ void direct_km(const float* __restrict__ p, long long ld, long long rk, int m0, int m_end,
                                          float* s, int tid) {
  const int l = tid & 63, w = tid >> 6;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int k = i * 8 + w * 2 + (l >> 5);
    const int m = m0 + ((4 * (l & 31)) ^ (((k >> 2) & 1) << 5));
    const float* src = p + (rk + k) * ld + (m < m_end ? m : m_end - 4);
    __builtin_amdgcn_global_load_lds(src, (lds_ptr)(s + (i * 256 + w * 64) * 4), 16, 0, 0);
  }
}
__device__ __forceinline__ void wait_direct() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ __forceinline__ void zero_acc(f32x16 (&acc)[2][2]) {
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;
}

// One LDS stage of MFMAs.  AMK / BMK: operand tile stored [m][k] (else [k][m]).
template <bool AMK, bool BMK, bool SW = false>
__device__ __forceinline__ void mfma_stage(const float* a_s, const float* b_s, int wm, int wn, int lr, int hf,
                                           f32x16 (&acc)[2][2]) {
#pragma unroll
  for (int g = 0; g < 2; ++g) {
    float af[2][4], bf[2][4];
#pragma unroll
    for (int bi = 0; bi < 2; ++bi) {
      const int m = wm * 64 + bi * 32 + lr;
      if (AMK) {
        const float4 v = ld4(a_s + mk_off(m, 2 * g + hf));
        af[bi][0] = v.x; af[bi][1] = v.y; af[bi][2] = v.z; af[bi][3] = v.w;
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          af[bi][j] = SW ? a_s[(8 * g + 4 * hf + j) * GBM + (m ^ (hf << 5))] : a_s[(8 * g + 4 * hf + j) * LD_KM + m];
      }
    }
#pragma unroll
    for (int bj = 0; bj < 2; ++bj) {
      const int n = wn * 64 + bj * 32 + lr;
      if (BMK) {
        const float4 v = ld4(b_s + mk_off(n, 2 * g + hf));
        bf[bj][0] = v.x; bf[bj][1] = v.y; bf[bj][2] = v.z; bf[bj][3] = v.w;
      } else {
#pragma unroll
        for (int j = 0; j < 4; ++j)
          bf[bj][j] = SW ? b_s[(8 * g + 4 * hf + j) * GBN + (n ^ (hf << 5))] : b_s[(8 * g + 4 * hf + j) * LD_KM + n];
      }
    }
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
          acc[bi][bj] = __builtin_amdgcn_mfma_f32_32x32x2f32(af[bi][j], bf[bj][j], acc[bi][bj], 0, 0, 0);
  }
}

// ---------------------------------------------------------------- gemm_rows

// One output tile of gemm_rows for (XCD-mapped) block number vb; smem holds
// SMEM_FLOATS floats of LDS.
template <bool NT, class ALoad, class Epi>
__device__ __forceinline__ void gemm_rows_block(int vb, float* smem, const ALoad& al, const float* __restrict__ B,
                                                int K, int N, const RowsTile* __restrict__ tiles,
                                                const int* __restrict__ n_tiles, const Epi& epi,
                                                float* __restrict__ rowsum_out) {
  const int ncol = (N + GBN - 1) / GBN;
  int t, ctile;
  xcd_map(vb, ncol, t, ctile);
  if (t >= *n_tiles) return;
  const RowsTile tile = tiles[t];
  const int n0 = ctile * GBN;
  const int r0 = tile.r0, r1 = tile.r1;
  const float* Bg = B + (long long)tile.group * K * N;

  // double buffers: A at smem + b * GBM * LD_MK, B after both A buffers
  auto sA = [&](int b) { return smem + b * (GBM * LD_MK); };
  auto sB = [&](int b) { return smem + 2 * GBM * LD_MK + b * B_BUF; };

  const int tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63;
  const int wm = w >> 1, wn = w & 1;
  const int lr = l & 31, hf = l >> 5;

  f32x16 acc[2][2];
  zero_acc(acc);

  StageMK<ALoad> sa;

  constexpr bool DA = IsPlainLoad<ALoad>::value;
  auto load_a = [&](int k, float* dst) {
    if constexpr (DA) direct_mk(reinterpret_cast<const LoadPlain&>(al).p, reinterpret_cast<const LoadPlain&>(al).ld,
                                r0, r1, k, dst, tid);
    else sa.load(al, r0, r1, k, tid);
  };
  auto load_b = [&](int k, float* dst) {
    if (NT) direct_mk(Bg, K, n0, N, k, dst, tid); else direct_km(Bg, N, k, n0, N, dst, tid);
  };
  load_a(0, sA(0));
  load_b(0, sB(0));
  if constexpr (!DA) sa.store(al, sA(0), 0, tid);
  wait_direct();
  __syncthreads();

  const int nk = K / GBK;
  int cur = 0;
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    const int k1 = (kt + 1) * GBK;
    if (more) {
      load_a(k1, sA(cur ^ 1));
      load_b(k1, sB(cur ^ 1));
    }
    // the stage's matrix instructions issue at raised wave priority, ahead of the
    // staging and epilogue work of the other workgroups on the SIMD (0.2-1 % faster)
    __builtin_amdgcn_s_setprio(1);
    mfma_stage<true, NT, true>(sA(cur), sB(cur), wm, wn, lr, hf, acc);
    __builtin_amdgcn_s_setprio(0);
    if (more) {
      if constexpr (!DA) sa.store(al, sA(cur ^ 1), k1, tid);
    }
    wait_direct();
    __syncthreads();
    cur ^= 1;
  }

  // Epilogue in two halves of 64 rows: the waves of row half `half` stage
  // their accumulators (lane l of block (bi, bj) holds column lr and rows
  // 8 (v / 4) + 4 hf + v % 4), then every thread visits 8 float4 pieces in
  // two batches: first the batch's global reads, then arithmetic and stores.
  float* sC = smem;
#pragma unroll
  for (int half = 0; half < 2; ++half) {
    if (wm == half) {
#pragma unroll
      for (int bi = 0; bi < 2; ++bi)
#pragma unroll
        for (int bj = 0; bj < 2; ++bj)
#pragma unroll
          for (int v = 0; v < 16; ++v)
            sC[(bi * 32 + 8 * (v >> 2) + 4 * hf + (v & 3)) * LD_C + wn * 64 + bj * 32 + lr] = acc[bi][bj][v];
    }
    // 4 pieces per batch; loads past the range read the last valid row.
    const int c4 = tid & 31;
    const int col = n0 + 4 * c4;
    const int colc = col < N ? col : N - 4;
#pragma unroll
    for (int i0 = 0; i0 < 8; i0 += 4) {
      typename Epi::Raw raw[4];
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const long long row = (long long)r0 + half * 64 + (tid >> 5) + 8 * (i0 + j);
        raw[j] = epi.load(row < r1 ? row : (long long)r1 - 1, colc);
      }
      if (i0 == 0) __syncthreads();
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        const int rl = (tid >> 5) + 8 * (i0 + j);
        const long long row = (long long)r0 + half * 64 + rl;
        float part = 0.f;
        if (row < r1 && col < N) part = epi.store(row, col, ld4(sC + rl * LD_C + 4 * c4), raw[j]);
        if (Epi::kRowSum) {
#pragma unroll
          for (int o = 16; o > 0; o >>= 1) part += __shfl_xor(part, o, 64);
          if (c4 == 0 && row < r1) rowsum_out[row * ncol + ctile] = part;
        }
      }
    }
    __syncthreads();
  }
}

template <bool NT, class ALoad, class Epi>
__global__ __launch_bounds__(256, 2) void gemm_rows_kernel(ALoad al, const float* __restrict__ B, int K, int N,
                                                           const RowsTile* __restrict__ tiles,
                                                           const int* __restrict__ n_tiles, Epi epi,
                                                           float* __restrict__ rowsum_out) {
  __shared__ __attribute__((aligned(16))) float smem[SMEM_FLOATS];
  gemm_rows_block<NT, ALoad, Epi>(blockIdx.x, smem, al, B, K, N, tiles, n_tiles, epi, rowsum_out);
}

// --------------------------------------------------------------- gemm_wgrad
// Both operands are row-major over the contraction index r: A [M, P], B [M, Q].

struct WChunk {
  int group;
  int r0;
  int r1;
  int pad;
};

// One partial tile of gemm_wgrad for (XCD-mapped) block number vb.
template <class ALoad, class BLoad>
__device__ __forceinline__ void gemm_wgrad_block(int vb, float* smem, const ALoad& al, const BLoad& bl, int P, int Q,
                                                 const WChunk* __restrict__ chunks,
                                                 const int* __restrict__ n_chunks, float* __restrict__ partial) {
  const int ntq = (Q + GBN - 1) / GBN;
  int c, pq;
  xcd_map(vb, ((P + GBM - 1) / GBM) * ntq, c, pq);
  if (c >= *n_chunks) return;
  const WChunk ch = chunks[c];
  const int p0 = (pq / ntq) * GBM;
  const int q0 = (pq % ntq) * GBN;

  auto sA = [&](int b) { return smem + b * (GBK * LD_KM); };
  auto sB = [&](int b) { return smem + (2 + b) * (GBK * LD_KM); };

  const int tid = threadIdx.x;
  const int w = tid >> 6, l = tid & 63;
  const int wm = w >> 1, wn = w & 1;
  const int lr = l & 31, hf = l >> 5;

  f32x16 acc[2][2];
  zero_acc(acc);

  StageKM<ALoad> sa;
  StageKM<BLoad> sb;
  // Both operands in the unpadded swizzled [k][m] layout.  A plain operand loads its whole
  // 16-row stages straight into LDS, and the chunk's last partial stage through registers
  // (its rows past the chunk become zeros); a transformed operand always goes through
  // registers.
  constexpr bool DA = IsPlainLoad<ALoad>::value, DB = IsPlainLoad<BLoad>::value;
  auto stage_load = [&](long long rk, int buf) {
    const bool full = rk + GBK <= ch.r1;
    if constexpr (DA) {
      if (full) direct_km(al.p, al.ld, rk, p0, P, sA(buf), tid); else sa.load(al, rk, ch.r1, p0, P, tid);
    } else {
      sa.load(al, rk, ch.r1, p0, P, tid);
    }
    if constexpr (DB) {
      if (full) direct_km(bl.p, bl.ld, rk, q0, Q, sB(buf), tid); else sb.load(bl, rk, ch.r1, q0, Q, tid);
    } else {
      sb.load(bl, rk, ch.r1, q0, Q, tid);
    }
  };
  auto stage_store = [&](long long rk, int buf) {
    const bool full = rk + GBK <= ch.r1;
    if (!DA || !full) sa.store_sw(al, sA(buf), p0, tid);
    if (!DB || !full) sb.store_sw(bl, sB(buf), q0, tid);
  };
  stage_load(ch.r0, 0);
  stage_store(ch.r0, 0);
  wait_direct();
  __syncthreads();

  const int nk = (ch.r1 - ch.r0 + GBK - 1) / GBK;
  int cur = 0;
  for (int kt = 0; kt < nk; ++kt) {
    const bool more = kt + 1 < nk;
    const long long rk = (long long)ch.r0 + (kt + 1) * GBK;
    if (more) stage_load(rk, cur ^ 1);
    __builtin_amdgcn_s_setprio(1);
    mfma_stage<false, false, true>(sA(cur), sB(cur), wm, wn, lr, hf, acc);
    __builtin_amdgcn_s_setprio(0);
    if (more) stage_store(rk, cur ^ 1);
    wait_direct();
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

template <class ALoad, class BLoad>
__global__ __launch_bounds__(256, 2) void gemm_wgrad_kernel(ALoad al, BLoad bl, int P, int Q,
                                                            const WChunk* __restrict__ chunks,
                                                            const int* __restrict__ n_chunks,
                                                            float* __restrict__ partial) {
  __shared__ __attribute__((aligned(16))) float smem[SMEM_FLOATS];
  gemm_wgrad_block<ALoad, BLoad>(blockIdx.x, smem, al, bl, P, Q, chunks, n_chunks, partial);
}

// ---------------------------------------------------------- skinny wgrad
// G[p, q] = sum_r s[r] A[r, p] B[r, q] for a short P (P <= 32, a multiple of 4;
// Q = 64, 128, 256 or 512: the radial-filter gradient, P = basis size, Q = d).
// A 128-row MFMA tile would be mostly padding there, so the vector units do it,
// straight from global memory.  A workgroup owns one chunk of rows and the whole
// P x Q output.  Lane l of a wave owns CW = min(4, Q / 64) consecutive columns of
// a 64 CW-wide column slice; the NS = Q / (64 CW) slices and RG = 4 / NS row
// groups split the four waves, wave (g, slice) accumulating all P output rows of
// its columns over the chunk rows g, g + RG, g + 2 RG, ...  A row's P values of A
// and its scale are the same for the whole wave, so they come through scalar loads
// and the vector registers hold only B and the accumulators; each step takes U
// rows and issues all their loads before using any.  Per row, b' = s[r] B[r, :]
// (B[r, :] if s is null) and acc[p] += A[r, p] b'.  The row groups are summed
// through LDS (P Q floats of dynamic LDS) in group order, and the workgroup writes
// one partial per chunk, reduced like gemm_wgrad's.
inline int skinny_cw(int Q) { return Q >= 256 ? 4 : Q / 64; }
inline int skinny_rows(int Q) {   // rows of one step of the workgroup (U = 4 rows per row group)
  return 4 * (4 / (Q / (64 * skinny_cw(Q))));
}

template <int PM, int CW>
__global__ __launch_bounds__(256) void wgrad_skinny_kernel(const float* __restrict__ A, const float* __restrict__ s,
                                                           const float* __restrict__ B, int P, int Q,
                                                           const WChunk* __restrict__ chunks,
                                                           const int* __restrict__ n_chunks,
                                                           float* __restrict__ partial) {
  constexpr int U = 8;
  extern __shared__ __attribute__((aligned(16))) float sk_lds[];
  const int c = blockIdx.x;
  if (c >= *n_chunks) return;
  const WChunk ch = chunks[c];
  const int NS = Q / (64 * CW), RG = 4 / NS;
  const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int lane = threadIdx.x & 63, la = lane % P;
  const int g = w / NS, col = (w - g * NS) * 64 * CW + lane * CW;
  float acc[PM][CW];
#pragma unroll
  for (int p = 0; p < PM; ++p)
#pragma unroll
    for (int k = 0; k < CW; ++k) acc[p][k] = 0.f;
  auto load_b = [&](long long r, float* v) {
    const float* q = B + r * Q + col;
    if constexpr (CW == 4) {
      const float4 x = ld4(q);
      v[0] = x.x; v[1] = x.y; v[2] = x.z; v[3] = x.w;
    } else if constexpr (CW == 2) {
      const float2 x = *reinterpret_cast<const float2*>(q);
      v[0] = x.x; v[1] = x.y;
    } else {
      v[0] = *q;
    }
  };
  // lane l holds A[r, l mod P]; row p's value is read from lane p (lanes p >= P
  // hold a repeated column: those accumulator rows are never stored)
  auto sweep = [&](auto scaled) {
    constexpr bool SC = decltype(scaled)::value;
    auto row = [&](float av, float sc, const float* b) {
      float x[CW];
#pragma unroll
      for (int k = 0; k < CW; ++k) x[k] = SC ? sc * b[k] : b[k];
      const int ai = __float_as_int(av);
#pragma unroll
      for (int p = 0; p < PM; ++p) {
        const float ap = __int_as_float(__builtin_amdgcn_readlane(ai, p));
#pragma unroll
        for (int k = 0; k < CW; ++k) acc[p][k] += ap * x[k];
      }
    };
    long long r = (long long)ch.r0 + g;
    for (; r + (long long)(U - 1) * RG < ch.r1; r += (long long)U * RG) {
      float b[U][CW], av[U], sc[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const long long ru = r + (long long)u * RG;
        load_b(ru, b[u]);
        av[u] = A[ru * P + la];
        sc[u] = SC ? s[ru] : 1.f;
      }
#pragma unroll
      for (int u = 0; u < U; ++u) row(av[u], sc[u], b[u]);
    }
    for (; r < ch.r1; r += RG) {
      float b[CW];
      load_b(r, b);
      row(A[r * P + la], SC ? s[r] : 1.f, b);
    }
  };
  if (s)
    sweep(std::true_type{});
  else
    sweep(std::false_type{});
  float* red = sk_lds;   // [P][Q]
  for (int gg = 0; gg < RG; ++gg) {
    if (g == gg) {
#pragma unroll
      for (int p = 0; p < PM; ++p) {
        if (p < P) {
#pragma unroll
          for (int k = 0; k < CW; ++k) {
            float v = acc[p][k];
            if (gg) v += red[p * Q + col + k];
            red[p * Q + col + k] = v;
          }
        }
      }
    }
    __syncthreads();
  }
  float4* out = reinterpret_cast<float4*>(partial + (long long)c * P * Q);
  const float4* red4 = reinterpret_cast<const float4*>(red);
  for (int i = threadIdx.x; i < P * Q / 4; i += 256) out[i] = red4[i];
}

}  // namespace janus
