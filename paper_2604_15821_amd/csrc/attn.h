// Multi-head self-attention over every atom's edge messages (paper Sec.
// "Multi-head self-attention": each edge of a neighbourhood attends to every
// edge of the same neighbourhood, cost m d sum_i |N(i)|^2).
//
// Per atom i with edges e in N(i) (contiguous rows rowptr[i] .. rowptr[i+1])
// and head a (32 columns of q, k, v = m Wqkv, row layout [q | k | v]):
//   s_el  = q_e . k_l / sqrt(32)
//   p_el  = u_l exp(s_el) / sum_j u_j exp(s_ej)        (u = edge envelope)
//   o_e   = sum_l p_el v_l
//   osum_i = sum_e u_e o_e                              (then u_i = h_i + osum_i Wo)
// Two kernel families run the four passes (forward, force backward, tangent,
// final backward), both on the matrix cores: neighbourhoods of up to
// kAttnMfmaN edges hold every 16-row tile of one (atom, head) in registers
// (below); larger ones, up to kAttnMaxN edges, sweep the tiles (attn_tiled.h).
// Per-query softmax statistics (max of s, Z = sum u exp(s - max)) are stored by
// the forward and reused by the three backward passes.  The neighbourhood limit
// is checked before the step.
#pragma once

#include "edge.h"

namespace janus {

constexpr int kAttnDh = 32;
constexpr int kAttnMaxN = 256;
constexpr int kAttnWaves = 4;   // waves per workgroup (256 threads)

__device__ __forceinline__ void ld32(const float* __restrict__ p, float* x) {
#pragma unroll
  for (int c = 0; c < kAttnDh; c += 4) {
    const float4 v = *reinterpret_cast<const float4*>(p + c);
    x[c] = v.x;
    x[c + 1] = v.y;
    x[c + 2] = v.z;
    x[c + 3] = v.w;
  }
}

// Four independent partial sums: a single 32-long chain of dependent multiply-adds
// leaves the vector unit waiting on each result.
__device__ __forceinline__ float dot32(const float* a, const float* b) {
  float s[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int c = 0; c < kAttnDh; ++c) s[c & 3] += a[c] * b[c];
  return (s[0] + s[1]) + (s[2] + s[3]);
}

constexpr float kAttnScale = 0.17677669529663687f;   // 1 / sqrt(32)

// Envelope of every edge: u(r/r_c) and du/dr, both zero from r = r_c on (an
// edge of a caller's list at or past the cutoff, a Verlet skin for example,
// then takes no attention weight, as in the basis).
__global__ void attn_env_kernel(const float4* __restrict__ geo, long long Ne, float rc, float* __restrict__ uu,
                                float* __restrict__ ud) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const double x = (double)geo[e].w / rc;
  double u = 0.0, du = 0.0;
  if (x < 1.0) {
    const double x2 = x * x, x5 = x2 * x2 * x, x6 = x5 * x;
    u = 1.0 - 28.0 * x6 + 48.0 * x6 * x - 21.0 * x6 * x2;
    du = -168.0 * x5 * (1.0 - x) * (1.0 - x);
  }
  uu[e] = (float)u;
  ud[e] = (float)(du / rc);
}

// Orders one wave's LDS writes before its later reads (and reads before later overwrites).
__device__ __forceinline__ void wave_sync() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
  __builtin_amdgcn_wave_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

// ------------------------------------------------------------ matrix-core kernels
// Neighbourhoods of at most kAttnMfmaN edges run on v_mfma_f32_16x16x4_f32, with the
// edges padded to 16-row tiles.  Lane l works on row i16 = l % 16 of a tile and
// slot j4 = l / 16 of the contraction; the 32 head columns are contracted in 8 steps
// with column 8*j4 + s at step s, so each lane reads 8 consecutive floats of a row.
// Scores are formed transposed (keys x queries): lane l then holds, for each pair of
// tiles, keys 4*j4 + r (r = 0..3) of one query i16 -- exactly the A operand of the
// following product with the values, so no data moves between the two products.
constexpr int kAttnMfmaN = 64;
constexpr int kAttnTiles = kAttnMfmaN / 16;
static_assert(kAttnMfmaN % 16 == 0 && kAttnTiles >= 1 && kAttnTiles <= 4, "the register-resident kernels exist for 1 to 4 tiles");

typedef float f32x4v __attribute__((ext_vector_type(4)));

__device__ __forceinline__ f32x4v mfma16(float a, float b, f32x4v c) {
  return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
}

// 8 floats of row `row` (clamped to the neighbourhood, zero past it) starting at column c0.
__device__ __forceinline__ void frag8(const float* __restrict__ base, long long ld, int e0, int n, int row, int c0,
                                      float* x) {
  const int rr = row < n ? row : n - 1;
  const float* p = base + (long long)(e0 + rr) * ld + c0;
  const float4 a = *reinterpret_cast<const float4*>(p), b = *reinterpret_cast<const float4*>(p + 4);
  const float z = row < n ? 1.f : 0.f;
  x[0] = z * a.x; x[1] = z * a.y; x[2] = z * a.z; x[3] = z * a.w;
  x[4] = z * b.x; x[5] = z * b.y; x[6] = z * b.z; x[7] = z * b.w;
}

// Sum over the 16 lanes i16 of each lane group (every lane gets its group's sum):
// DPP quad_perm 1032, quad_perm 2301, half-row mirror, row mirror.
template <int CTRL>
__device__ __forceinline__ float attn_dpp_add(float v) {
  return v + __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), CTRL, 0xF, 0xF, true));
}
__device__ __forceinline__ float sum_i16(float v) {
  v = attn_dpp_add<0xB1>(v);
  v = attn_dpp_add<0x4E>(v);
  v = attn_dpp_add<0x141>(v);
  return attn_dpp_add<0x140>(v);
}

// Sum (or max) over the four lane groups j4 of a value owned by row i16.
__device__ __forceinline__ float sum_j4(float v) {
  v += __shfl_xor(v, 16, 64);
  return v + __shfl_xor(v, 32, 64);
}
__device__ __forceinline__ float max_j4(float v) {
  v = fmaxf(v, __shfl_xor(v, 16, 64));
  return fmaxf(v, __shfl_xor(v, 32, 64));
}

// Phase 1 on matrix cores for the atoms whose neighbourhood spans NT 16-row tiles
// (NT = 1 also takes the atoms without edges); one instance per NT keeps the register
// use of the small neighbourhoods small.  Same outputs as attn_fwd_tiled_kernel.
template <int NT>
__global__ __launch_bounds__(64 * kAttnWaves) void attn_fwd_mfma_kernel(
    const int* __restrict__ rowptr, const float* __restrict__ QKV, const float* __restrict__ uu, int N, int d, int H,
    float* __restrict__ stats, float* __restrict__ osum) {
  const long long ld = 3LL * d;
  const int i16 = threadIdx.x & 15, j4 = (threadIdx.x >> 4) & 3;
  // one wave per (atom, head)
  JANUS_WAVE_LOOP(item, (long long)N * H) {
    const int i = (int)(item / H), a = (int)(item - (long long)i * H);
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n == 0 && NT == 1) {
      if ((threadIdx.x & 63) < kAttnDh) osum[(long long)i * d + a * kAttnDh + (threadIdx.x & 63)] = 0.f;
      continue;
    }
    if ((n + 15) >> 4 != NT) continue;
    constexpr int nt = NT;
    {
      const int cq = a * kAttnDh, ck = d + a * kAttnDh, cv = 2 * d + a * kAttnDh;
      // every load of the head first: q and k fragments, the value columns and envelope
      // weights of the rows kt*16 + 4*j4 + r this lane feeds to the value product (the
      // same rows give the query weights of the output tile)
      float qf[NT][8], kf[NT][8], v0[NT][4], v1[NT][4], uk[NT][4];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        if (t >= nt) break;
        frag8(QKV, ld, e0, n, t * 16 + i16, cq + 8 * j4, qf[t]);
        frag8(QKV, ld, e0, n, t * 16 + i16, ck + 8 * j4, kf[t]);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = t * 16 + 4 * j4 + r;
          const int kk = key < n ? key : n - 1;
          const float* vr = QKV + (long long)(e0 + kk) * ld + cv + i16;
          v0[t][r] = vr[0];
          v1[t][r] = vr[16];
          uk[t][r] = key < n ? uu[e0 + kk] : 0.f;
        }
      }
      // transposed scores per (key tile, query tile); the contraction step is outermost so
      // the tile accumulators are independent
      f32x4v S[NT][NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int u = 0; u < NT; ++u) S[t][u] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 8; ++st)
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int qt = 0; qt < NT; ++qt)
            if (kt < nt && qt < nt) S[kt][qt] = mfma16(kf[kt][st], qf[qt][st], S[kt][qt]);
      // softmax over the keys of each query (query = qt*16 + i16; keys kt*16 + 4*j4 + r)
#pragma unroll
      for (int qt = 0; qt < NT; ++qt) {
        if (qt >= nt) break;
        float M = -INFINITY;
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
          if (kt >= nt) break;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = kt * 16 + 4 * j4 + r;
            const float sv = key < n ? S[kt][qt][r] * kAttnScale : -INFINITY;
            S[kt][qt][r] = sv;
            M = fmaxf(M, sv);
          }
        }
        M = max_j4(M);
        float Z = 0.f;
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
          if (kt >= nt) break;
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float pv = uk[kt][r] * __expf(S[kt][qt][r] - M);
            S[kt][qt][r] = pv;
            Z += pv;
          }
        }
        Z = sum_j4(Z);
        const float iZ = 1.f / Z;
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
          if (kt >= nt) break;
#pragma unroll
          for (int r = 0; r < 4; ++r) S[kt][qt][r] *= iZ;
        }
        const int q = qt * 16 + i16;
        if (j4 == 0 && q < n) {
          stats[((long long)(e0 + q) * H + a) * 2] = M;
          stats[((long long)(e0 + q) * H + a) * 2 + 1] = Z;
        }
      }
      // o = p v for every (query tile, 16-column tile), key steps outermost so the eight
      // accumulators are independent; osum = sum over queries of u_q o_q
      f32x4v O[NT][2];
#pragma unroll
      for (int qt = 0; qt < NT; ++qt) O[qt][0] = O[qt][1] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kt = 0; kt < NT; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
          for (int qt = 0; qt < NT; ++qt)
            if (kt < nt && qt < nt) {
              O[qt][0] = mfma16(S[kt][qt][r], v0[kt][r], O[qt][0]);
              O[qt][1] = mfma16(S[kt][qt][r], v1[kt][r], O[qt][1]);
            }
      float col0 = 0.f, col1 = 0.f;
#pragma unroll
      for (int qt = 0; qt < NT; ++qt) {
        if (qt >= nt) break;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          col0 += uk[qt][r] * O[qt][0][r];
          col1 += uk[qt][r] * O[qt][1][r];
        }
      }
      col0 = sum_j4(col0);
      col1 = sum_j4(col1);
      if (j4 == 0) {
        osum[(long long)i * d + cq + i16] = col0;
        osum[(long long)i * d + cq + 16 + i16] = col1;
      }
    }
  }
}

// Phase 3 on matrix cores for the atoms whose neighbourhood spans NT 16-row tiles
// (NT = 1 also takes the atoms without edges), one wave per (atom, head); same output as
// attn_tan_tiled_kernel.  Transposed score tiles S = k.q and Sh = k.qh + kh.q give, per
// (key, query), p = u_k E and pz = p sh + uh_k E with E = exp(s - M_q)/Z_q (stored
// statistics); then oh = pz v - (sum pz) o + p vh with o = p v, three value products
// chained on the probability tiles as in the forward.
template <int NT>
__global__ __launch_bounds__(64 * kAttnWaves) void attn_tan_mfma_kernel(
    const int* __restrict__ rowptr, const float* __restrict__ QKV, const float* __restrict__ QKVh,
    const float* __restrict__ uu, const float* __restrict__ ud, const float* __restrict__ rt,
    const float* __restrict__ stats, int N, int d, int H, float* __restrict__ osumh) {
  const long long ld = 3LL * d;
  const int i16 = threadIdx.x & 15, j4 = (threadIdx.x >> 4) & 3;
  JANUS_WAVE_LOOP(item, (long long)N * H) {
    const int i = (int)(item / H), a = (int)(item - (long long)i * H);
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n == 0 && NT == 1) {
      if ((threadIdx.x & 63) < kAttnDh) osumh[(long long)i * d + a * kAttnDh + (threadIdx.x & 63)] = 0.f;
      continue;
    }
    if ((n + 15) >> 4 != NT) continue;
    const int cq = a * kAttnDh, ck = d + a * kAttnDh, cv = 2 * d + a * kAttnDh;
    // scores and their tangents, transposed (key tile, query tile)
    f32x4v S[NT][NT], Sh[NT][NT];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int u = 0; u < NT; ++u) S[t][u] = Sh[t][u] = f32x4v{0.f, 0.f, 0.f, 0.f};
    {
      float qf[NT][8], kf[NT][8];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        frag8(QKV, ld, e0, n, t * 16 + i16, cq + 8 * j4, qf[t]);
        frag8(QKV, ld, e0, n, t * 16 + i16, ck + 8 * j4, kf[t]);
      }
#pragma unroll
      for (int st = 0; st < 8; ++st)
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int qt = 0; qt < NT; ++qt) S[kt][qt] = mfma16(kf[kt][st], qf[qt][st], S[kt][qt]);
      float hf[NT][8];
#pragma unroll
      for (int t = 0; t < NT; ++t) frag8(QKVh, ld, e0, n, t * 16 + i16, cq + 8 * j4, hf[t]);   // qh
#pragma unroll
      for (int st = 0; st < 8; ++st)
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int qt = 0; qt < NT; ++qt) Sh[kt][qt] = mfma16(kf[kt][st], hf[qt][st], Sh[kt][qt]);
#pragma unroll
      for (int t = 0; t < NT; ++t) frag8(QKVh, ld, e0, n, t * 16 + i16, ck + 8 * j4, hf[t]);   // kh
#pragma unroll
      for (int st = 0; st < 8; ++st)
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int qt = 0; qt < NT; ++qt) Sh[kt][qt] = mfma16(hf[kt][st], qf[qt][st], Sh[kt][qt]);
    }
    // per-key weights of the rows kt*16 + 4*j4 + r (also the output rows' query weights)
    float uk[NT][4], uhk[NT][4];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = t * 16 + 4 * j4 + r;
        const int kk = key < n ? key : n - 1;
        uk[t][r] = key < n ? uu[e0 + kk] : 0.f;
        uhk[t][r] = key < n ? ud[e0 + kk] * rt[e0 + kk] : 0.f;
      }
    // p (into S) and pz (into Sh); s1 = sum over keys of pz, per query
    float s1[NT];
#pragma unroll
    for (int qt = 0; qt < NT; ++qt) {
      const int q = qt * 16 + i16;
      const long long sq = ((long long)(e0 + (q < n ? q : n - 1)) * H + a) * 2;
      const float M = stats[sq], iZ = 1.f / stats[sq + 1];
      float sum = 0.f;
#pragma unroll
      for (int kt = 0; kt < NT; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float E = __expf(S[kt][qt][r] * kAttnScale - M) * iZ;
          const float p = uk[kt][r] * E;
          const float pz = p * Sh[kt][qt][r] * kAttnScale + uhk[kt][r] * E;
          S[kt][qt][r] = p;
          Sh[kt][qt][r] = pz;
          sum += pz;
        }
      s1[qt] = sum_j4(sum);
    }
    // value products: o = p v, oz = pz v, ov = p vh, per (query tile, 16-column tile)
    f32x4v O[NT][2], OZ[NT][2], OV[NT][2];
#pragma unroll
    for (int qt = 0; qt < NT; ++qt)
#pragma unroll
      for (int ct = 0; ct < 2; ++ct) O[qt][ct] = OZ[qt][ct] = OV[qt][ct] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int kt = 0; kt < NT; ++kt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kt * 16 + 4 * j4 + r;
        const long long row = (long long)(e0 + (key < n ? key : n - 1)) * ld;
        const float v0 = QKV[row + cv + i16], v1 = QKV[row + cv + 16 + i16];
        const float w0 = QKVh[row + cv + i16], w1 = QKVh[row + cv + 16 + i16];
#pragma unroll
        for (int qt = 0; qt < NT; ++qt) {
          O[qt][0] = mfma16(S[kt][qt][r], v0, O[qt][0]);
          O[qt][1] = mfma16(S[kt][qt][r], v1, O[qt][1]);
          OZ[qt][0] = mfma16(Sh[kt][qt][r], v0, OZ[qt][0]);
          OZ[qt][1] = mfma16(Sh[kt][qt][r], v1, OZ[qt][1]);
          OV[qt][0] = mfma16(S[kt][qt][r], w0, OV[qt][0]);
          OV[qt][1] = mfma16(S[kt][qt][r], w1, OV[qt][1]);
        }
      }
    // osumh = sum over queries of u_q oh_q + uh_q o_q, oh = oz - s1 o + ov (rows qt*16 + 4*j4 + r)
    float col0 = 0.f, col1 = 0.f;
#pragma unroll
    for (int qt = 0; qt < NT; ++qt)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const float s1r = __shfl(s1[qt], 4 * j4 + r, 64);   // s1 of query qt*16 + 4*j4 + r
        const float u = uk[qt][r], uh = uhk[qt][r];
        col0 += u * (OZ[qt][0][r] - s1r * O[qt][0][r] + OV[qt][0][r]) + uh * O[qt][0][r];
        col1 += u * (OZ[qt][1][r] - s1r * O[qt][1][r] + OV[qt][1][r]) + uh * O[qt][1][r];
      }
    col0 = sum_j4(col0);
    col1 = sum_j4(col1);
    if (j4 == 0) {
      osumh[(long long)i * d + cq + i16] = col0;
      osumh[(long long)i * d + cq + 16 + i16] = col1;
    }
  }
}

// Phase 2 on matrix cores for the atoms whose neighbourhood spans NT 16-row tiles, one
// wave per (atom, head); same outputs as attn_bwd_tiled_kernel: the envelope
// terms of dE/dr go to rbh [(e H + a)] (query term cw_e plus key term kl_e of head a)
// and attn_rbar_kernel adds them to rbar.  Transposed score tiles (key x query) give
// p, cw and zb = u_q p (w_k - cw_q) in the A-operand layout of qb = zb k, and the per-key
// sums Pu = sum_q u_q p (vb = Pu ob) and kl = sum_q u_q E (w_k - cw_q) by adding over
// the 16 query lanes; each zb tile is transposed through LDS (1 KB per wave) into the
// layout of kb = zb^T q.
template <int NT>
__global__ __launch_bounds__(64 * kAttnWaves, NT <= 3 ? 2 : 1) void attn_bwd_mfma_kernel(
    const int* __restrict__ rowptr, const float* __restrict__ QKV, const float* __restrict__ uu,
    const float* __restrict__ stats, const float* __restrict__ ob, int N, int d, int H, float* __restrict__ QKVb,
    float* __restrict__ rbh) {
  constexpr int LT = 20;   // row stride of a transposed tile (floats)
  __shared__ __attribute__((aligned(16))) float s_tr[kAttnWaves][16 * LT];
  float* tz = s_tr[threadIdx.x >> 6];
  const long long ld = 3LL * d;
  const int i16 = threadIdx.x & 15, j4 = (threadIdx.x >> 4) & 3;
  JANUS_WAVE_LOOP(item, (long long)N * H) {
    const int i = (int)(item / H), a = (int)(item - (long long)i * H);
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n == 0 || (n + 15) >> 4 != NT) continue;
    const int cq = a * kAttnDh, ck = d + a * kAttnDh, cv = 2 * d + a * kAttnDh;
    float qf[NT][8], kf[NT][8];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      frag8(QKV, ld, e0, n, t * 16 + i16, cq + 8 * j4, qf[t]);
      frag8(QKV, ld, e0, n, t * 16 + i16, ck + 8 * j4, kf[t]);
    }
    // ob columns 8 j4 .. 8 j4 + 7 and w_k = ob . v_k for the rows t*16 + i16 (every j4 lane)
    float obf[8];
    {
      const float* po = ob + (long long)i * d + cq + 8 * j4;
      const float4 x = *reinterpret_cast<const float4*>(po), y = *reinterpret_cast<const float4*>(po + 4);
      obf[0] = x.x; obf[1] = x.y; obf[2] = x.z; obf[3] = x.w;
      obf[4] = y.x; obf[5] = y.y; obf[6] = y.z; obf[7] = y.w;
    }
    float wrow[NT], urow[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      float vf[8];
      frag8(QKV, ld, e0, n, t * 16 + i16, cv + 8 * j4, vf);
      float s = 0.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) s += obf[c] * vf[c];
      wrow[t] = sum_j4(s);
      const int row = t * 16 + i16;
      urow[t] = row < n ? uu[e0 + row] : 0.f;
    }
    // ---- transposed tiles: lane holds (key kt*16 + 4 j4 + r, query qt*16 + i16)
    {
      f32x4v S[NT][NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int u = 0; u < NT; ++u) S[t][u] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int st = 0; st < 8; ++st)
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int qt = 0; qt < NT; ++qt) S[kt][qt] = mfma16(kf[kt][st], qf[qt][st], S[kt][qt]);
      float uk[NT][4], wk[NT][4];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          uk[t][r] = __shfl(urow[t], 4 * j4 + r, 64);   // u of key t*16 + 4 j4 + r
          wk[t][r] = __shfl(wrow[t], 4 * j4 + r, 64);
        }
      // per key kt*16 + 4 j4 + r, partial over this lane's queries: sum u_q p, and
      // kl = sum u_q E (w_k - cw_q)
      float pu[NT][4], kl[NT][4], cw[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int r = 0; r < 4; ++r) pu[t][r] = kl[t][r] = 0.f;
#pragma unroll
      for (int qt = 0; qt < NT; ++qt) {
        const int q = qt * 16 + i16;
        const long long sq = ((long long)(e0 + (q < n ? q : n - 1)) * H + a) * 2;
        const float M = stats[sq], iZ = 1.f / stats[sq + 1];
        float c = 0.f;
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float E = __expf(S[kt][qt][r] * kAttnScale - M) * iZ;
            S[kt][qt][r] = E;
            c += uk[kt][r] * E * wk[kt][r];
          }
        cw[qt] = sum_j4(c);
        // zb = u_q p (w_k - cw_q), in place
        const float uq = urow[qt];
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const float E = S[kt][qt][r], p = uk[kt][r] * E, dw = wk[kt][r] - cw[qt];
            pu[kt][r] += uq * p;
            kl[kt][r] += uq * E * dw;
            S[kt][qt][r] = uq * p * dw;
          }
      }
      // qb = (1/sqrt 32) zb k: lane holds (query qt*16 + 4 j4 + r, column ct*16 + i16)
      {
        f32x4v QB[NT][2];
#pragma unroll
        for (int qt = 0; qt < NT; ++qt) QB[qt][0] = QB[qt][1] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int key = kt * 16 + 4 * j4 + r;
            const long long row = (long long)(e0 + (key < n ? key : n - 1)) * ld;
            const float k0 = QKV[row + ck + i16], k1 = QKV[row + ck + 16 + i16];
#pragma unroll
            for (int qt = 0; qt < NT; ++qt) {
              QB[qt][0] = mfma16(S[kt][qt][r], k0, QB[qt][0]);
              QB[qt][1] = mfma16(S[kt][qt][r], k1, QB[qt][1]);
            }
          }
#pragma unroll
        for (int qt = 0; qt < NT; ++qt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int q = qt * 16 + 4 * j4 + r;
            if (q < n) {
              float* o = QKVb + (long long)(e0 + q) * ld + cq;
              o[i16] = kAttnScale * QB[qt][0][r];
              o[16 + i16] = kAttnScale * QB[qt][1][r];
            }
          }
      }
      // ---- per-key sums over the 16 query lanes: lane (i16, j4) then holds those of keys
      // kt*16 + 4 j4 + r.  vb = Pu ob: lane i16 writes key 4 j4 + i16 / 4, columns
      // 8 (i16 % 4) ..; envelope term of edge e = 4 j4 + i16 (lanes i16 < 4): cw_e + kl_e
      const int rs = i16 >> 2, cg = i16 & 3;
      float obw[8];
      {
        const float* po = ob + (long long)i * d + cq + 8 * cg;
        const float4 x = *reinterpret_cast<const float4*>(po), y = *reinterpret_cast<const float4*>(po + 4);
        obw[0] = x.x; obw[1] = x.y; obw[2] = x.z; obw[3] = x.w;
        obw[4] = y.x; obw[5] = y.y; obw[6] = y.z; obw[7] = y.w;
      }
#pragma unroll
      for (int kt = 0; kt < NT; ++kt) {
        float P = 0.f, K = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float v1 = sum_i16(pu[kt][r]), v2 = sum_i16(kl[kt][r]);
          P = rs == r ? v1 : P;
          K = cg == r ? v2 : K;
        }
        const int key = kt * 16 + 4 * j4 + rs;
        if (key < n) {
          float* o = QKVb + (long long)(e0 + key) * ld + cv + 8 * cg;
          *reinterpret_cast<float4*>(o) = make_float4(P * obw[0], P * obw[1], P * obw[2], P * obw[3]);
          *reinterpret_cast<float4*>(o + 4) = make_float4(P * obw[4], P * obw[5], P * obw[6], P * obw[7]);
        }
        const float c = __shfl(cw[kt], 4 * j4 + cg, 64);   // cw of row kt*16 + 4 j4 + cg
        const int row = kt * 16 + 4 * j4 + cg;
        if (i16 < 4 && row < n) rbh[(long long)(e0 + row) * H + a] = c + K;
      }
      // ---- kb = (1/sqrt 32) zb^T q: each zb tile transposed through LDS, lane (i16, j4)
      // receiving (query qt*16 + 4 j4 + r, key kt*16 + i16); lane holds (key kt*16 + 4 j4 + r,
      // column ct*16 + i16) of kb
      f32x4v KB[NT][2];
#pragma unroll
      for (int kt = 0; kt < NT; ++kt) KB[kt][0] = KB[kt][1] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int qt = 0; qt < NT; ++qt) {
        float zt[NT][4];
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
          *reinterpret_cast<float4*>(tz + i16 * LT + 4 * j4) =
              make_float4(S[kt][qt][0], S[kt][qt][1], S[kt][qt][2], S[kt][qt][3]);
          wave_sync();
#pragma unroll
          for (int r = 0; r < 4; ++r) zt[kt][r] = tz[(4 * j4 + r) * LT + i16];
          wave_sync();
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = qt * 16 + 4 * j4 + r;
          const long long row = (long long)(e0 + (q < n ? q : n - 1)) * ld;
          const float x0 = QKV[row + cq + i16], x1 = QKV[row + cq + 16 + i16];
#pragma unroll
          for (int kt = 0; kt < NT; ++kt) {
            KB[kt][0] = mfma16(zt[kt][r], x0, KB[kt][0]);
            KB[kt][1] = mfma16(zt[kt][r], x1, KB[kt][1]);
          }
        }
      }
#pragma unroll
      for (int kt = 0; kt < NT; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt * 16 + 4 * j4 + r;
          if (key < n) {
            float* o = QKVb + (long long)(e0 + key) * ld + ck;
            o[i16] = kAttnScale * KB[kt][0][r];
            o[16 + i16] = kAttnScale * KB[kt][1][r];
          }
        }
    }
  }
}

// Phase 4 on matrix cores for the atoms whose neighbourhood spans NT 16-row tiles, one
// wave per (atom, head); same output as attn_rev_tiled_kernel.  Per row t*16 + i16 (every j4
// lane): u, uh = u' rt, a = alpha.v + beta.vh and b = beta.v (8-column partial dots
// added over the four lane groups), the query's softmax statistics.  Transposed tiles
// (key x query) of s and sh give the per-query sums am, bm, zm, pbz and SP, then zb and
// zhb in the A-operand layout of qb = zb k + zhb kh.  The same tiles give the per-key
// sums S1 = sum u_q p, S2 = sum uh_q p + u_q (pz - p zm) of vb = S1 alpha + S2 beta (and,
// with POS, sum_q zb) by adding over the 16 query lanes, and each (zb, zhb) tile pair is
// transposed through LDS (2 KB per wave) into the A-operand layout of
// kb = zb^T q + zhb^T qh, so no score tile is formed twice.
template <int NT, bool POS>
__global__ __launch_bounds__(64 * kAttnWaves, NT <= 3 && !POS ? 2 : 1) void attn_rev_mfma_kernel(
    const int* __restrict__ rowptr, const float* __restrict__ QKV, const float* __restrict__ QKVh,
    const float* __restrict__ uu, const float* __restrict__ ud, const float* __restrict__ rt,
    const float* __restrict__ stats, const float* __restrict__ alpha, const float* __restrict__ beta, int N, int d,
    int H, float* __restrict__ QKVa, float* __restrict__ rlh) {
  // multiply-adds are fused only inside one expression: the instance that also forms the
  // log-u adjoints (POS) then computes every other output with the same roundings
#pragma clang fp contract(on)
  constexpr int LT = 20;   // row stride of a transposed tile (floats)
  __shared__ __attribute__((aligned(16))) float s_tr[kAttnWaves][2][16 * LT];
  float* tz = s_tr[threadIdx.x >> 6][0];
  float* th = s_tr[threadIdx.x >> 6][1];
  const long long ld = 3LL * d;
  const int i16 = threadIdx.x & 15, j4 = (threadIdx.x >> 4) & 3;
  JANUS_WAVE_LOOP(item, (long long)N * H) {
    const int i = (int)(item / H), a = (int)(item - (long long)i * H);
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n == 0 || (n + 15) >> 4 != NT) continue;
    const int cq = a * kAttnDh, ck = d + a * kAttnDh, cv = 2 * d + a * kAttnDh;
    float alf[8], bef[8];
    {
      const float* pa = alpha + (long long)i * d + cq + 8 * j4;
      const float* pb = beta + (long long)i * d + cq + 8 * j4;
#pragma unroll
      for (int c = 0; c < 8; c += 4) {
        const float4 x = *reinterpret_cast<const float4*>(pa + c), y = *reinterpret_cast<const float4*>(pb + c);
        alf[c] = x.x; alf[c + 1] = x.y; alf[c + 2] = x.z; alf[c + 3] = x.w;
        bef[c] = y.x; bef[c + 1] = y.y; bef[c + 2] = y.z; bef[c + 3] = y.w;
      }
    }
    // per row t*16 + i16
    float urow[NT], uhrow[NT], arow[NT], brow[NT], mrow[NT], izrow[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      float vf[8], wf[8];
      frag8(QKV, ld, e0, n, t * 16 + i16, cv + 8 * j4, vf);
      frag8(QKVh, ld, e0, n, t * 16 + i16, cv + 8 * j4, wf);
      float sa = 0.f, sb = 0.f;
#pragma unroll
      for (int c = 0; c < 8; ++c) {
        sa += alf[c] * vf[c] + bef[c] * wf[c];
        sb += bef[c] * vf[c];
      }
      arow[t] = sum_j4(sa);
      brow[t] = sum_j4(sb);
      const int row = t * 16 + i16;
      const int rr = row < n ? row : n - 1;
      urow[t] = row < n ? uu[e0 + rr] : 0.f;
      uhrow[t] = row < n ? ud[e0 + rr] * rt[e0 + rr] : 0.f;
      const long long sq = ((long long)(e0 + rr) * H + a) * 2;
      mrow[t] = stats[sq];
      izrow[t] = 1.f / stats[sq + 1];
    }
    float lq[POS ? NT : 1];            // with POS: query part of the adjoint of log u, row t*16 + i16
    // per key kt*16 + 4 j4 + r, partial over this lane's queries: S1, S2 (and sum_q zb)
    float c1[NT][4], c2[NT][4], c3[POS ? NT : 1][4];
#pragma unroll
    for (int t = 0; t < NT; ++t)
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        c1[t][r] = c2[t][r] = 0.f;
        if (POS) c3[t][r] = 0.f;
      }
    // ---- transposed tiles: lane holds (key kt*16 + 4 j4 + r, query qt*16 + i16)
    {
      f32x4v S[NT][NT], Sh[NT][NT];
#pragma unroll
      for (int t = 0; t < NT; ++t)
#pragma unroll
        for (int u = 0; u < NT; ++u) S[t][u] = Sh[t][u] = f32x4v{0.f, 0.f, 0.f, 0.f};
      {
        float qf[NT][8], kf[NT][8], hf[NT][8];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
          frag8(QKV, ld, e0, n, t * 16 + i16, cq + 8 * j4, qf[t]);
          frag8(QKV, ld, e0, n, t * 16 + i16, ck + 8 * j4, kf[t]);
        }
#pragma unroll
        for (int st = 0; st < 8; ++st)
#pragma unroll
          for (int kt = 0; kt < NT; ++kt)
#pragma unroll
            for (int qt = 0; qt < NT; ++qt) S[kt][qt] = mfma16(kf[kt][st], qf[qt][st], S[kt][qt]);
#pragma unroll
        for (int t = 0; t < NT; ++t) frag8(QKVh, ld, e0, n, t * 16 + i16, cq + 8 * j4, hf[t]);   // qh
#pragma unroll
        for (int st = 0; st < 8; ++st)
#pragma unroll
          for (int kt = 0; kt < NT; ++kt)
#pragma unroll
            for (int qt = 0; qt < NT; ++qt) Sh[kt][qt] = mfma16(kf[kt][st], hf[qt][st], Sh[kt][qt]);
#pragma unroll
        for (int t = 0; t < NT; ++t) frag8(QKVh, ld, e0, n, t * 16 + i16, ck + 8 * j4, hf[t]);   // kh
#pragma unroll
        for (int st = 0; st < 8; ++st)
#pragma unroll
          for (int kt = 0; kt < NT; ++kt)
#pragma unroll
            for (int qt = 0; qt < NT; ++qt) Sh[kt][qt] = mfma16(hf[kt][st], qf[qt][st], Sh[kt][qt]);
      }
      // p into S, pz into Sh; per-query sums
#pragma unroll
      for (int qt = 0; qt < NT; ++qt) {
        float am = 0.f, bm = 0.f, zm = 0.f, pbz = 0.f;
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int src = 4 * j4 + r;
            const float uk = __shfl(urow[kt], src, 64), uhk = __shfl(uhrow[kt], src, 64);
            const float ak = __shfl(arow[kt], src, 64), bk = __shfl(brow[kt], src, 64);
            const float E = __expf(S[kt][qt][r] * kAttnScale - mrow[qt]) * izrow[qt];
            const float p = uk * E;
            const float pz = p * Sh[kt][qt][r] * kAttnScale + uhk * E;
            S[kt][qt][r] = p;
            Sh[kt][qt][r] = pz;
            am += p * ak;
            bm += p * bk;
            zm += pz;
            pbz += pz * bk;
          }
        am = sum_j4(am);
        bm = sum_j4(bm);
        zm = sum_j4(zm);
        pbz = sum_j4(pbz);
        const float ue = urow[qt], uh = uhrow[qt];
        const float SP = ue * (am + pbz - 2.f * zm * bm) + uh * bm;
        if (POS) lq[qt] = ue * (am + pbz - zm * bm) + uh * bm;   // query part of the log-u adjoint
        // zb into S, zhb into Sh; this query's terms of the per-key sums
#pragma unroll
        for (int kt = 0; kt < NT; ++kt)
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const int src = 4 * j4 + r;
            const float ak = __shfl(arow[kt], src, 64), bk = __shfl(brow[kt], src, 64);
            const float p = S[kt][qt][r], pz = Sh[kt][qt][r];
            c1[kt][r] += ue * p;
            c2[kt][r] += uh * p + ue * (pz - p * zm);
            const float zb = ue * (p * ak + bk * (pz - p * zm) - pz * bm) + uh * p * bk - p * SP;
            S[kt][qt][r] = zb;
            Sh[kt][qt][r] = ue * p * (bk - bm);
            if (POS) c3[kt][r] += zb;   // key part of the log-u adjoint
          }
      }
      // qb = (1/sqrt 32)(zb k + zhb kh): lane holds (query qt*16 + 4 j4 + r, column ct*16 + i16)
      f32x4v QB[NT][2];
#pragma unroll
      for (int qt = 0; qt < NT; ++qt) QB[qt][0] = QB[qt][1] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int kt = 0; kt < NT; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt * 16 + 4 * j4 + r;
          const long long row = (long long)(e0 + (key < n ? key : n - 1)) * ld;
          const float k0 = QKV[row + ck + i16], k1 = QKV[row + ck + 16 + i16];
          const float h0 = QKVh[row + ck + i16], h1 = QKVh[row + ck + 16 + i16];
#pragma unroll
          for (int qt = 0; qt < NT; ++qt) {
            QB[qt][0] = mfma16(S[kt][qt][r], k0, QB[qt][0]);
            QB[qt][1] = mfma16(S[kt][qt][r], k1, QB[qt][1]);
            QB[qt][0] = mfma16(Sh[kt][qt][r], h0, QB[qt][0]);
            QB[qt][1] = mfma16(Sh[kt][qt][r], h1, QB[qt][1]);
          }
        }
#pragma unroll
      for (int qt = 0; qt < NT; ++qt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = qt * 16 + 4 * j4 + r;
          if (q < n) {
            float* o = QKVa + (long long)(e0 + q) * ld + cq;
            o[i16] = kAttnScale * QB[qt][0][r];
            o[16 + i16] = kAttnScale * QB[qt][1][r];
          }
        }
      // ---- per-key sums over the 16 query lanes: lane (i16, j4) then holds those of keys
      // kt*16 + 4 j4 + r; lane i16 writes key 4 j4 + i16 / 4, columns 8 (i16 % 4) ..
      const int rs = i16 >> 2, cg = i16 & 3;
      float alw[8], bew[8];
      {
        const float* pa = alpha + (long long)i * d + cq + 8 * cg;
        const float* pb = beta + (long long)i * d + cq + 8 * cg;
#pragma unroll
        for (int c = 0; c < 8; c += 4) {
          const float4 x = *reinterpret_cast<const float4*>(pa + c), y = *reinterpret_cast<const float4*>(pb + c);
          alw[c] = x.x; alw[c + 1] = x.y; alw[c + 2] = x.z; alw[c + 3] = x.w;
          bew[c] = y.x; bew[c + 1] = y.y; bew[c + 2] = y.z; bew[c + 3] = y.w;
        }
      }
#pragma unroll
      for (int kt = 0; kt < NT; ++kt) {
        float A1 = 0.f, A2 = 0.f, L = 0.f;
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const float v1 = sum_i16(c1[kt][r]), v2 = sum_i16(c2[kt][r]);
          A1 = rs == r ? v1 : A1;
          A2 = rs == r ? v2 : A2;
          if (POS) {
            const float v3 = sum_i16(c3[kt][r]);
            L = cg == r ? v3 : L;
          }
        }
        const int key = kt * 16 + 4 * j4 + rs;
        if (key < n) {
          // vb = S1 alpha + S2 beta
          float* o = QKVa + (long long)(e0 + key) * ld + cv + 8 * cg;
          *reinterpret_cast<float4*>(o) = make_float4(A1 * alw[0] + A2 * bew[0], A1 * alw[1] + A2 * bew[1],
                                                      A1 * alw[2] + A2 * bew[2], A1 * alw[3] + A2 * bew[3]);
          *reinterpret_cast<float4*>(o + 4) = make_float4(A1 * alw[4] + A2 * bew[4], A1 * alw[5] + A2 * bew[5],
                                                          A1 * alw[6] + A2 * bew[6], A1 * alw[7] + A2 * bew[7]);
        }
        if (POS) {
          // adjoint of log u_e, edge e = kt*16 + 4 j4 + cg: key part + query part (row e's lane)
          const float q = __shfl(lq[kt], 4 * j4 + cg, 64);
          const int row = kt * 16 + 4 * j4 + cg;
          if (i16 < 4 && row < n) rlh[(long long)(e0 + row) * H + a] = L + q;
        }
      }
      // ---- kb = (1/sqrt 32)(zb^T q + zhb^T qh): each (zb, zhb) tile pair transposed through
      // LDS, lane (i16, j4) receiving (query qt*16 + 4 j4 + r, key kt*16 + i16); lane holds
      // (key kt*16 + 4 j4 + r, column ct*16 + i16) of kb
      f32x4v KB[NT][2];
#pragma unroll
      for (int kt = 0; kt < NT; ++kt) KB[kt][0] = KB[kt][1] = f32x4v{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int qt = 0; qt < NT; ++qt) {
        float zt[NT][4], ht[NT][4];
#pragma unroll
        for (int kt = 0; kt < NT; ++kt) {
          *reinterpret_cast<float4*>(tz + i16 * LT + 4 * j4) =
              make_float4(S[kt][qt][0], S[kt][qt][1], S[kt][qt][2], S[kt][qt][3]);
          *reinterpret_cast<float4*>(th + i16 * LT + 4 * j4) =
              make_float4(Sh[kt][qt][0], Sh[kt][qt][1], Sh[kt][qt][2], Sh[kt][qt][3]);
          wave_sync();
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            zt[kt][r] = tz[(4 * j4 + r) * LT + i16];
            ht[kt][r] = th[(4 * j4 + r) * LT + i16];
          }
          wave_sync();
        }
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = qt * 16 + 4 * j4 + r;
          const long long row = (long long)(e0 + (q < n ? q : n - 1)) * ld;
          const float x0 = QKV[row + cq + i16], x1 = QKV[row + cq + 16 + i16];
          const float h0 = QKVh[row + cq + i16], h1 = QKVh[row + cq + 16 + i16];
#pragma unroll
          for (int kt = 0; kt < NT; ++kt) {
            KB[kt][0] = mfma16(zt[kt][r], x0, KB[kt][0]);
            KB[kt][1] = mfma16(zt[kt][r], x1, KB[kt][1]);
            KB[kt][0] = mfma16(ht[kt][r], h0, KB[kt][0]);
            KB[kt][1] = mfma16(ht[kt][r], h1, KB[kt][1]);
          }
        }
      }
#pragma unroll
      for (int kt = 0; kt < NT; ++kt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt * 16 + 4 * j4 + r;
          if (key < n) {
            float* o = QKVa + (long long)(e0 + key) * ld + ck;
            o[i16] = kAttnScale * KB[kt][0][r];
            o[16 + i16] = kAttnScale * KB[kt][1][r];
          }
        }
    }
  }
}

// dE/dr of the edges of the atoms the matrix-core phase-2 kernel took (n <= nmax):
// rbar_e += u'(r_e) sum over heads a (in order) of rbh[e H + a].  One wave per atom.
__global__ void attn_rbar_kernel(const int* __restrict__ rowptr, const float* __restrict__ ud,
                                 const float* __restrict__ rbh, int N, int H, int nmax, float* __restrict__ rbar,
                                 float* __restrict__ rbs) {
  JANUS_WAVE_LOOP(i, N) {
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n > nmax) continue;
    for (int j = l; j < n; j += kWave) {
      const long long e = e0 + j;
      float s = 0.f;
      for (int a = 0; a < H; ++a) s += rbh[e * H + a];
      rbar[e] += ud[e] * s;
      if (rbs) rbs[e] = s;   // dE/du_e of this block, kept for the loss gradient in positions
    }
  }
}

// Loss gradient in positions through the attention envelope, one block: with
// lu = log u(r / r_c) and its tangent rho = (d lu / dr) rt, the final backward gives
// L_e = d(loss)/d lu_e (rlh, per head) and the force backward R_e = d(loss)/d rho_e =
// u_e dE/du_e (rbs, the head sum, times u); then
//   rpos_e += L_e (d lu / dr) + R_e rt_e (d2 lu / dr2)
//          = L_e u'/u + rbs_e rt_e (u'' - u'^2 / u),
// in float64 from r_e; edges at or past r_c (u = 0) take no part.
__global__ void attn_pos_kernel(const float4* __restrict__ geo, long long Ne, int H, float rc,
                                const float* __restrict__ rlh, const float* __restrict__ rbs,
                                const float* __restrict__ rt, float* __restrict__ rpos) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const double x = (double)geo[e].w / rc;
  if (!(x < 1.0)) return;
  const double x2 = x * x, x4 = x2 * x2, x5 = x4 * x, x6 = x5 * x;
  const double u = 1.0 - 28.0 * x6 + 48.0 * x6 * x - 21.0 * x6 * x2;
  const double u1 = -168.0 * x5 * (1.0 - x) * (1.0 - x) / rc;
  const double u2 = (-840.0 * x4 + 2016.0 * x5 - 1176.0 * x6) / ((double)rc * rc);
  double L = 0.0;
  for (int a = 0; a < H; ++a) L += rlh[e * H + a];
  rpos[e] += (float)(L * u1 / u + (double)rbs[e] * (double)rt[e] * (u2 - u1 * u1 / u));
}

// Messages per edge from the expert slots: out_e = sum_c Y[pos[e, c]] (already gated).
template <int VPL, int KC>
__global__ void edge_sum_kernel(const int* __restrict__ pos, const float* __restrict__ Y, long long Ne, int d,
                                float* __restrict__ out) {
  JANUS_WAVE_LOOP(e, Ne) {
    float y[VPL];
    sum_slots<VPL, KC>(Y, pos, e, d, l, y);
    st_row<VPL>(out + e * d, l, y);
  }
}

// Slot rows of a per-edge adjoint: out[pos[e, c]] = (g_ec) src_e.
template <int VPL, int KC>
__global__ void edge_gather_kernel(const int* __restrict__ pos, const float* __restrict__ gate,
                                   const float* __restrict__ src, long long Ne, int d, float* __restrict__ out) {
  JANUS_WAVE_LOOP(e, Ne) {
    float s[VPL];
    ld_row<VPL>(src + e * d, l, s);
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      const long long f = e * KC + c;
      const float g = gate ? gate[f] : 1.f;
      float o[VPL];
#pragma unroll
      for (int v = 0; v < VPL; ++v) o[v] = g * s[v];
      st_row<VPL>(out + (long long)pos[f] * d, l, o);
    }
  }
}

// Phase 3 per edge: mh_e = sum_c g_ec Ybt[pos[e, c]] (tangent of the message) and the gate
// adjoints g3_ec = Ybt[pos[e, c]] . mbar_e (mbar = the phase-2 adjoint of the message).
template <int VPL, int KC>
__global__ void edge_combine_p3_kernel(const int* __restrict__ pos, const float* __restrict__ gate,
                                       const float* __restrict__ Ybt, const float* __restrict__ mbar, long long Ne,
                                       int d, float* __restrict__ g3, float* __restrict__ mh) {
  JANUS_WAVE_LOOP(e, Ne) {
    float mb[VPL], acc[VPL];
    ld_row<VPL>(mbar + e * d, l, mb);
    zero_row<VPL>(acc);
    float s[KC];
#pragma unroll
    for (int c = 0; c < KC; ++c) {
      float y[VPL];
      ld_row<VPL>(Ybt + (long long)pos[e * KC + c] * d, l, y);
      const float g = gate[e * KC + c];
      s[c] = 0.f;
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        s[c] += y[v] * mb[v];
        acc[v] += g * y[v];
      }
    }
#pragma unroll
    for (int c = 0; c < KC; ++c) s[c] = wave_sum(s[c]);
    if (l == 0) {
#pragma unroll
      for (int c = 0; c < KC; ++c) g3[e * KC + c] = s[c];
    }
    st_row<VPL>(mh + e * d, l, acc);
  }
}

// Largest neighbourhood: flag[1] |= 1 when an atom has more than kAttnMaxN edges.
__global__ void attn_degree_check_kernel(const int* __restrict__ rowptr, int N, int* __restrict__ flag) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < N && rowptr[i + 1] - rowptr[i] > kAttnMaxN) atomicOr(flag + 1, 1);
}

}  // namespace janus
