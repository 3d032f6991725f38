// Matrix-core passes of the neighbourhood self-attention for neighbourhoods of
// kAttnMfmaN + 1 .. kAttnMaxN edges (the register-resident kernels of attn.h take
// the smaller ones).  One wave per (atom, head) walks 16-row tiles: a sweep over
// query tiles (keys of each tile pair visited in turn) forms every per-query sum
// and the products of the scores with key or value rows, a sweep over key tiles
// (queries visited in turn) forms the per-key sums; scores are recomputed in each
// sweep from the stored softmax statistics.  Score tiles come in two orientations
// on v_mfma_f32_16x16x4_f32:
//   keys x queries (score_kq): lane (i16, j4) holds the scores of query i16 with
//     keys 4 j4 + r, r = 0..3 -- the A operand of a product contracted over keys;
//   queries x keys (score_qk): lane (i16, j4) holds key i16 with queries 4 j4 + r
//     -- the A operand of a product contracted over queries.
// Per-row scalars that one sweep produces and the other reads live in LDS (per
// wave, kAttnMaxN entries each).  The arithmetic per (query, key) pair is that of
// the register-resident kernels (attn.h).
#pragma once

#include "attn.h"

namespace janus {

// Head widths of the tiled kernels: DH = 32, 64 or 128 columns; lane group j4 holds
// CG = DH / 4 consecutive columns of a row (the contraction's step st takes column
// CG j4 + st), and a product with DH output columns has OT = DH / 16 column tiles.
template <int DH>
struct AttnW {
  static_assert(DH == 32 || DH == 64 || DH == 128, "head widths of 32, 64 or 128 columns");
  static constexpr int CG = DH / 4;
  static constexpr int OT = DH / 16;
};
constexpr float attn_scale(int dh) {   // 1 / sqrt(dh)
  return dh == 32 ? 0.17677669529663687f : dh == 64 ? 0.125f : 0.08838834764831845f;
}

// CG floats of row `row` (clamped to the neighbourhood, zero past it) starting at column c0.
template <int CG>
__device__ __forceinline__ void fragw(const float* __restrict__ base, long long ld, int e0, int n, int row, int c0,
                                      float (&x)[CG]) {
  const int rr = row < n ? row : n - 1;
  const float* p = base + (long long)(e0 + rr) * ld + c0;
  const float z = row < n ? 1.f : 0.f;
#pragma unroll
  for (int c = 0; c < CG; c += 4) {
    const float4 a = *reinterpret_cast<const float4*>(p + c);
    x[c] = z * a.x;
    x[c + 1] = z * a.y;
    x[c + 2] = z * a.z;
    x[c + 3] = z * a.w;
  }
}

template <int CG>
__device__ __forceinline__ f32x4v score_kq(const float (&kf)[CG], const float (&qf)[CG], f32x4v s) {
#pragma unroll
  for (int st = 0; st < CG; ++st) s = mfma16(kf[st], qf[st], s);
  return s;
}
template <int CG>
__device__ __forceinline__ f32x4v score_qk(const float (&qf)[CG], const float (&kf)[CG], f32x4v s) {
#pragma unroll
  for (int st = 0; st < CG; ++st) s = mfma16(qf[st], kf[st], s);
  return s;
}
__device__ __forceinline__ f32x4v zero4() { return f32x4v{0.f, 0.f, 0.f, 0.f}; }

// B operand of a product contracted over rows: columns c0 + 16 t + i16 (t < OT) of
// row `row` of the neighbourhood (clamped to it; the A operand is zero past n).
template <int OT>
__device__ __forceinline__ void colsw(const float* __restrict__ base, long long ld, int e0, int n, int row, int c0,
                                      int i16, float (&x)[OT]) {
  const float* p = base + (long long)(e0 + (row < n ? row : n - 1)) * ld + c0 + i16;
#pragma unroll
  for (int t = 0; t < OT; ++t) x[t] = p[16 * t];
}

// Dot product of two DH-column rows, 32 columns at a time.
template <int DH>
__device__ __forceinline__ float dot_rows(const float* __restrict__ a, const float* __restrict__ b) {
  float x[kAttnDh], y[kAttnDh];
  ld32(a, x);
  ld32(b, y);
  float s = dot32(x, y);
#pragma unroll
  for (int c0 = kAttnDh; c0 < DH; c0 += kAttnDh) {
    ld32(a + c0, x);
    ld32(b + c0, y);
    s += dot32(x, y);
  }
  return s;
}

// Per-row scalars of one neighbourhood staged in the wave's LDS region before its
// sweeps, so the tile loops read them from LDS: the envelope u, its tangent
// uh = u' rt (when uh is wanted) and the softmax statistics M, 1/Z of head a (when
// stats is given).  Call between wave_sync()s.
__device__ __forceinline__ void stage_rows(int e0, int n, int H, int a, const float* __restrict__ uu,
                                           const float* __restrict__ ud, const float* __restrict__ rt,
                                           const float* __restrict__ stats, float* su, float* suh, float* sM,
                                           float* siZ, int l) {
  for (int k = l; k < n; k += 64) {
    su[k] = uu[e0 + k];
    if (suh) suh[k] = ud[e0 + k] * rt[e0 + k];
    if (sM) {
      const long long sq = ((long long)(e0 + k) * H + a) * 2;
      sM[k] = stats[sq];
      siZ[k] = 1.f / stats[sq + 1];
    }
  }
}

// Phase 1 for the neighbourhoods of more than nmin edges (nmin = kAttnMfmaN beside the
// register-resident kernels, -1 for heads wider than 32 columns, where these kernels
// take every atom).  Same outputs as attn_fwd_mfma_kernel: stats (max s, Z) per
// (query, head) and osum_i.
template <int DH>
__global__ __launch_bounds__(64 * kAttnWaves) void attn_fwd_tiled_kernel(
    const int* __restrict__ rowptr, const float* __restrict__ QKV, const float* __restrict__ uu, int N, int d, int H,
    int nmin, float* __restrict__ stats, float* __restrict__ osum) {
  constexpr int CG = AttnW<DH>::CG, OT = AttnW<DH>::OT;
  constexpr float scale = attn_scale(DH);
  __shared__ float s_u[kAttnWaves][kAttnMaxN];
  float* su = s_u[threadIdx.x >> 6];
  const long long ld = 3LL * d;
  const int i16 = threadIdx.x & 15, j4 = (threadIdx.x >> 4) & 3;
  JANUS_WAVE_LOOP(item, (long long)N * H) {
    const int i = (int)(item / H), a = (int)(item - (long long)i * H);
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n <= nmin) continue;
    const int nt = (n + 15) >> 4;
    const int cq = a * DH, ck = d + a * DH, cv = 2 * d + a * DH;
    wave_sync();
    stage_rows(e0, n, H, a, uu, nullptr, nullptr, nullptr, su, nullptr, nullptr, nullptr, l);
    wave_sync();
    float col[OT];
#pragma unroll
    for (int t = 0; t < OT; ++t) col[t] = 0.f;
    for (int qt = 0; qt < nt; ++qt) {
      float qf[CG];
      fragw<CG>(QKV, ld, e0, n, qt * 16 + i16, cq + CG * j4, qf);
      // max over the keys of query qt*16 + i16
      float M = -INFINITY;
      for (int kt = 0; kt < nt; ++kt) {
        float kf[CG];
        fragw<CG>(QKV, ld, e0, n, kt * 16 + i16, ck + CG * j4, kf);
        const f32x4v S = score_kq<CG>(kf, qf, zero4());
#pragma unroll
        for (int r = 0; r < 4; ++r)
          if (kt * 16 + 4 * j4 + r < n) M = fmaxf(M, S[r] * scale);
      }
      M = max_j4(M);
      // Z and the unnormalised o = sum_l u_l exp(s - M) v_l (rows: queries qt*16 + 4*j4 + r)
      float Z = 0.f;
      f32x4v O[OT];
#pragma unroll
      for (int t = 0; t < OT; ++t) O[t] = zero4();
      for (int kt = 0; kt < nt; ++kt) {
        float kf[CG];
        fragw<CG>(QKV, ld, e0, n, kt * 16 + i16, ck + CG * j4, kf);
        const f32x4v S = score_kq<CG>(kf, qf, zero4());
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt * 16 + 4 * j4 + r;
          const float u = key < n ? su[key] : 0.f;
          const float pv = u * __expf(S[r] * scale - M);
          Z += pv;
          float v[OT];
          colsw<OT>(QKV, ld, e0, n, key, cv, i16, v);
#pragma unroll
          for (int t = 0; t < OT; ++t) O[t] = mfma16(pv, v[t], O[t]);
        }
      }
      Z = sum_j4(Z);
      const int qq = qt * 16 + i16;
      if (j4 == 0 && qq < n) {
        stats[((long long)(e0 + qq) * H + a) * 2] = M;
        stats[((long long)(e0 + qq) * H + a) * 2 + 1] = Z;
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = qt * 16 + 4 * j4 + r;
        const float Zq = __shfl(Z, 4 * j4 + r, 64);
        const float w = q < n ? su[q] / Zq : 0.f;
#pragma unroll
        for (int t = 0; t < OT; ++t) col[t] += w * O[t][r];
      }
    }
#pragma unroll
    for (int t = 0; t < OT; ++t) col[t] = sum_j4(col[t]);
    if (j4 == 0) {
#pragma unroll
      for (int t = 0; t < OT; ++t) osum[(long long)i * d + cq + 16 * t + i16] = col[t];
    }
  }
}

// Phase 3 (tangent) for the neighbourhoods of more than nmin edges; same output as
// attn_tan_mfma_kernel: osumh_i = sum_q u_q oh_q + uh_q o_q,
// oh_q = sum_l pz_ql v_l - (sum_l pz_ql) o_q + sum_l p_ql vh_l.
template <int DH>
__global__ __launch_bounds__(64 * kAttnWaves) void attn_tan_tiled_kernel(
    const int* __restrict__ rowptr, const float* __restrict__ QKV, const float* __restrict__ QKVh,
    const float* __restrict__ uu, const float* __restrict__ ud, const float* __restrict__ rt,
    const float* __restrict__ stats, int N, int d, int H, int nmin, float* __restrict__ osumh) {
  constexpr int CG = AttnW<DH>::CG, OT = AttnW<DH>::OT;
  constexpr float scale = attn_scale(DH);
  __shared__ float s_u[kAttnWaves][2][kAttnMaxN];
  float* su = s_u[threadIdx.x >> 6][0];
  float* suh = s_u[threadIdx.x >> 6][1];
  const long long ld = 3LL * d;
  const int i16 = threadIdx.x & 15, j4 = (threadIdx.x >> 4) & 3;
  JANUS_WAVE_LOOP(item, (long long)N * H) {
    const int i = (int)(item / H), a = (int)(item - (long long)i * H);
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n <= nmin) continue;
    const int nt = (n + 15) >> 4;
    const int cq = a * DH, ck = d + a * DH, cv = 2 * d + a * DH;
    wave_sync();
    stage_rows(e0, n, H, a, uu, ud, rt, nullptr, su, suh, nullptr, nullptr, l);
    wave_sync();
    float col[OT];
#pragma unroll
    for (int t = 0; t < OT; ++t) col[t] = 0.f;
    for (int qt = 0; qt < nt; ++qt) {
      float qf[CG], qhf[CG];
      fragw<CG>(QKV, ld, e0, n, qt * 16 + i16, cq + CG * j4, qf);
      fragw<CG>(QKVh, ld, e0, n, qt * 16 + i16, cq + CG * j4, qhf);
      const int qq = qt * 16 + i16, qc = qq < n ? qq : n - 1;
      const long long sq = ((long long)(e0 + qc) * H + a) * 2;
      const float M = stats[sq], iZ = 1.f / stats[sq + 1];
      f32x4v A1[OT], A2[OT], A3[OT];
#pragma unroll
      for (int t = 0; t < OT; ++t) A1[t] = A2[t] = A3[t] = zero4();
      float s1 = 0.f;
      for (int kt = 0; kt < nt; ++kt) {
        float kf[CG], khf[CG];
        fragw<CG>(QKV, ld, e0, n, kt * 16 + i16, ck + CG * j4, kf);
        fragw<CG>(QKVh, ld, e0, n, kt * 16 + i16, ck + CG * j4, khf);
        const f32x4v S = score_kq<CG>(kf, qf, zero4());
        const f32x4v Sh = score_kq<CG>(khf, qf, score_kq<CG>(kf, qhf, zero4()));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt * 16 + 4 * j4 + r;
          const int kk = key < n ? key : n - 1;
          const float uk = key < n ? su[kk] : 0.f, uhk = key < n ? suh[kk] : 0.f;
          const float E = __expf(S[r] * scale - M) * iZ;
          const float p = uk * E;
          const float pz = p * Sh[r] * scale + uhk * E;
          s1 += pz;
          float v[OT], w[OT];
          colsw<OT>(QKV, ld, e0, n, key, cv, i16, v);
          colsw<OT>(QKVh, ld, e0, n, key, cv, i16, w);
#pragma unroll
          for (int t = 0; t < OT; ++t) A1[t] = mfma16(pz, v[t], A1[t]);
#pragma unroll
          for (int t = 0; t < OT; ++t) A2[t] = mfma16(p, v[t], A2[t]);
#pragma unroll
          for (int t = 0; t < OT; ++t) A3[t] = mfma16(p, w[t], A3[t]);
        }
      }
      s1 = sum_j4(s1);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = qt * 16 + 4 * j4 + r;
        const float s1r = __shfl(s1, 4 * j4 + r, 64);
        const float u = q < n ? su[q] : 0.f, uh = q < n ? suh[q] : 0.f;
#pragma unroll
        for (int t = 0; t < OT; ++t) col[t] += u * (A1[t][r] - s1r * A2[t][r] + A3[t][r]) + uh * A2[t][r];
      }
    }
#pragma unroll
    for (int t = 0; t < OT; ++t) col[t] = sum_j4(col[t]);
    if (j4 == 0) {
#pragma unroll
      for (int t = 0; t < OT; ++t) osumh[(long long)i * d + cq + 16 * t + i16] = col[t];
    }
  }
}

// Phase 2 (force backward) for the neighbourhoods of more than nmin edges; same
// outputs as attn_bwd_mfma_kernel: QKVb rows (qb | kb | vb) and rbh[e H + a] = cw_e + kl_e.
//   w_l = ob . v_l, cw_q = sum_l p_ql w_l, qb_q = u_q (sum_l p w_l k_l - cw_q sum_l p k_l) / sqrt(DH),
//   t_ql = u_q E_ql (w_l - cw_q), kl_l = sum_q t_ql, kb_l = u_l sum_q t_ql q_q / sqrt(DH),
//   vb_l = (sum_q u_q u_l E_ql) ob.
template <int DH>
__global__ __launch_bounds__(64 * kAttnWaves) void attn_bwd_tiled_kernel(
    const int* __restrict__ rowptr, const float* __restrict__ QKV, const float* __restrict__ uu,
    const float* __restrict__ stats, const float* __restrict__ ob, int N, int d, int H, int nmin,
    float* __restrict__ QKVb, float* __restrict__ rbh) {
  constexpr int CG = AttnW<DH>::CG, OT = AttnW<DH>::OT;
  constexpr float scale = attn_scale(DH);
  __shared__ float s_sc[kAttnWaves][5][kAttnMaxN];
  float* wk = s_sc[threadIdx.x >> 6][0];
  float* cw = s_sc[threadIdx.x >> 6][1];
  float* su = s_sc[threadIdx.x >> 6][2];
  float* sM = s_sc[threadIdx.x >> 6][3];
  float* siZ = s_sc[threadIdx.x >> 6][4];
  const long long ld = 3LL * d;
  const int i16 = threadIdx.x & 15, j4 = (threadIdx.x >> 4) & 3;
  JANUS_WAVE_LOOP(item, (long long)N * H) {
    const int i = (int)(item / H), a = (int)(item - (long long)i * H);
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n <= nmin) continue;
    const int nt = (n + 15) >> 4;
    const int cq = a * DH, ck = d + a * DH, cv = 2 * d + a * DH;
    const float* obh = ob + (long long)i * d + cq;
    wave_sync();
    stage_rows(e0, n, H, a, uu, nullptr, nullptr, stats, su, nullptr, sM, siZ, l);
    for (int k = l; k < n; k += 64) wk[k] = dot_rows<DH>(obh, QKV + (long long)(e0 + k) * ld + cv);
    wave_sync();
    // queries: cw and qb
    for (int qt = 0; qt < nt; ++qt) {
      float qf[CG];
      fragw<CG>(QKV, ld, e0, n, qt * 16 + i16, cq + CG * j4, qf);
      const int qq = qt * 16 + i16, qc = qq < n ? qq : n - 1;
      const long long sq = ((long long)(e0 + qc) * H + a) * 2;
      const float M = stats[sq], iZ = 1.f / stats[sq + 1];
      f32x4v A1[OT], A2[OT];
#pragma unroll
      for (int t = 0; t < OT; ++t) A1[t] = A2[t] = zero4();
      float sw = 0.f;
      for (int kt = 0; kt < nt; ++kt) {
        float kf[CG];
        fragw<CG>(QKV, ld, e0, n, kt * 16 + i16, ck + CG * j4, kf);
        const f32x4v S = score_kq<CG>(kf, qf, zero4());
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt * 16 + 4 * j4 + r;
          const int kk = key < n ? key : n - 1;
          const float p = (key < n ? su[kk] : 0.f) * __expf(S[r] * scale - M) * iZ;
          const float pw = p * wk[kk];
          sw += pw;
          float kc[OT];
          colsw<OT>(QKV, ld, e0, n, key, ck, i16, kc);
#pragma unroll
          for (int t = 0; t < OT; ++t) A1[t] = mfma16(pw, kc[t], A1[t]);
#pragma unroll
          for (int t = 0; t < OT; ++t) A2[t] = mfma16(p, kc[t], A2[t]);
        }
      }
      sw = sum_j4(sw);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = qt * 16 + 4 * j4 + r;
        const float swq = __shfl(sw, 4 * j4 + r, 64);
        if (q < n) {
          const float uq = su[q] * scale;
          float* out = QKVb + (long long)(e0 + q) * ld + cq + i16;
#pragma unroll
          for (int t = 0; t < OT; ++t) out[16 * t] = uq * (A1[t][r] - swq * A2[t][r]);
        }
      }
      if (j4 == 0 && qq < n) cw[qq] = sw;
    }
    wave_sync();
    // keys: kb, vb and the key term of rbh
    float obc[OT];
#pragma unroll
    for (int t = 0; t < OT; ++t) obc[t] = obh[16 * t + i16];
    for (int kt = 0; kt < nt; ++kt) {
      float kf[CG];
      fragw<CG>(QKV, ld, e0, n, kt * 16 + i16, ck + CG * j4, kf);
      const int kn = kt * 16 + i16, kc = kn < n ? kn : n - 1;
      const float uk = kn < n ? su[kc] : 0.f, w = wk[kc];
      f32x4v KB[OT];
#pragma unroll
      for (int t = 0; t < OT; ++t) KB[t] = zero4();
      float Pu = 0.f, kl = 0.f;
      for (int qt = 0; qt < nt; ++qt) {
        float qf[CG];
        fragw<CG>(QKV, ld, e0, n, qt * 16 + i16, cq + CG * j4, qf);
        const f32x4v S = score_qk<CG>(qf, kf, zero4());
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = qt * 16 + 4 * j4 + r;
          const int qc = q < n ? q : n - 1;
          const float uq = q < n ? su[qc] : 0.f;
          const float E = __expf(S[r] * scale - sM[qc]) * siZ[qc];
          const float t = uq * E * (w - cw[qc]);
          kl += t;
          Pu += uq * uk * E;
          float qv[OT];
          colsw<OT>(QKV, ld, e0, n, q, cq, i16, qv);
#pragma unroll
          for (int c = 0; c < OT; ++c) KB[c] = mfma16(uk * t, qv[c], KB[c]);
        }
      }
      kl = sum_j4(kl);
      Pu = sum_j4(Pu);
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kt * 16 + 4 * j4 + r;
        const float Pur = __shfl(Pu, 4 * j4 + r, 64);
        if (key < n) {
          float* out = QKVb + (long long)(e0 + key) * ld;
#pragma unroll
          for (int t = 0; t < OT; ++t) out[ck + 16 * t + i16] = KB[t][r] * scale;
#pragma unroll
          for (int t = 0; t < OT; ++t) out[cv + 16 * t + i16] = Pur * obc[t];
        }
      }
      if (j4 == 0 && kn < n) rbh[(long long)(e0 + kn) * H + a] = cw[kn] + kl;
    }
  }
}

// Phase 4 (final backward through the forward and its tangent) for the neighbourhoods
// of more than nmin edges; same output as attn_rev_mfma_kernel.  alpha_i is the
// adjoint of osum_i, beta_i that of the tangent osumh_i; per query the adjoints of o_q
// and oh_q are u_q alpha + uh_q beta and u_q beta.  With a_l = alpha.v_l + beta.vh_l,
// b_l = beta.v_l and, per query, am = sum p a, bm = sum p b, zm = sum pz, pbz = sum pz b,
// SP = u_q (am + pbz - 2 zm bm) + uh_q bm:
//   zb_ql  = u_q (p a_l + b_l (pz - p zm) - pz bm) + uh_q p b_l - p SP   (adjoint of s_ql)
//   zhb_ql = u_q p (b_l - bm)                                            (adjoint of sh_ql)
//   qb_q = sum_l (zb k_l + zhb kh_l) / sqrt(DH),  kb_l = sum_q (zb q_q + zhb qh_q) / sqrt(DH),
//   vb_l = alpha sum_q u_q p + beta sum_q (uh_q p + u_q (pz - p zm)).
// QKVa rows get (qb | kb | vb), the adjoints of the primal q, k, v.  With rlh (the loss
// gradient in positions) it also gets, per (edge, head), the adjoint of log u_e:
// the sum over queries of zb_qe (key part) plus u_e (am + pbz - zm bm) + uh_e bm (query
// part, u_e alpha.o_e + u_e beta.oh_e + uh_e beta.o_e).
template <int DH>
__global__ __launch_bounds__(64 * kAttnWaves) void attn_rev_tiled_kernel(
    const int* __restrict__ rowptr, const float* __restrict__ QKV, const float* __restrict__ QKVh,
    const float* __restrict__ uu, const float* __restrict__ ud, const float* __restrict__ rt,
    const float* __restrict__ stats, const float* __restrict__ alpha, const float* __restrict__ beta, int N, int d,
    int H, int nmin, float* __restrict__ QKVa, float* __restrict__ rlh) {
  constexpr int CG = AttnW<DH>::CG, OT = AttnW<DH>::OT;
  constexpr float scale = attn_scale(DH);
  __shared__ float s_sc[kAttnWaves][10][kAttnMaxN];
  float* lq_ = s_sc[threadIdx.x >> 6][9];
  float* su = s_sc[threadIdx.x >> 6][5];
  float* suh = s_sc[threadIdx.x >> 6][6];
  float* sM = s_sc[threadIdx.x >> 6][7];
  float* siZ = s_sc[threadIdx.x >> 6][8];
  float* sa = s_sc[threadIdx.x >> 6][0];
  float* sb = s_sc[threadIdx.x >> 6][1];
  float* bm_ = s_sc[threadIdx.x >> 6][2];
  float* zm_ = s_sc[threadIdx.x >> 6][3];
  float* sp_ = s_sc[threadIdx.x >> 6][4];
  const long long ld = 3LL * d;
  const int i16 = threadIdx.x & 15, j4 = (threadIdx.x >> 4) & 3;
  JANUS_WAVE_LOOP(item, (long long)N * H) {
    const int i = (int)(item / H), a = (int)(item - (long long)i * H);
    const int e0 = rowptr[i], n = rowptr[i + 1] - e0;
    if (n <= nmin) continue;
    const int nt = (n + 15) >> 4;
    const int cq = a * DH, ck = d + a * DH, cv = 2 * d + a * DH;
    const float* al = alpha + (long long)i * d + cq;
    const float* be = beta + (long long)i * d + cq;
    wave_sync();
    stage_rows(e0, n, H, a, uu, ud, rt, stats, su, suh, sM, siZ, l);
    // per key: a_l = alpha . v_l + beta . vh_l, b_l = beta . v_l
    for (int k = l; k < n; k += 64) {
      const float* v = QKV + (long long)(e0 + k) * ld + cv;
      const float* vh = QKVh + (long long)(e0 + k) * ld + cv;
      sa[k] = dot_rows<DH>(al, v) + dot_rows<DH>(be, vh);
      sb[k] = dot_rows<DH>(be, v);
    }
    wave_sync();
    // queries: per-query sums, then qb
    for (int qt = 0; qt < nt; ++qt) {
      float qf[CG], qhf[CG];
      fragw<CG>(QKV, ld, e0, n, qt * 16 + i16, cq + CG * j4, qf);
      fragw<CG>(QKVh, ld, e0, n, qt * 16 + i16, cq + CG * j4, qhf);
      const int qq = qt * 16 + i16, qc = qq < n ? qq : n - 1;
      const long long sq = ((long long)(e0 + qc) * H + a) * 2;
      const float M = stats[sq], iZ = 1.f / stats[sq + 1];
      float am = 0.f, bm = 0.f, zm = 0.f, pbz = 0.f;
      for (int kt = 0; kt < nt; ++kt) {
        float kf[CG], khf[CG];
        fragw<CG>(QKV, ld, e0, n, kt * 16 + i16, ck + CG * j4, kf);
        fragw<CG>(QKVh, ld, e0, n, kt * 16 + i16, ck + CG * j4, khf);
        const f32x4v S = score_kq<CG>(kf, qf, zero4());
        const f32x4v Sh = score_kq<CG>(khf, qf, score_kq<CG>(kf, qhf, zero4()));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt * 16 + 4 * j4 + r;
          const int kk = key < n ? key : n - 1;
          const float uk = key < n ? su[kk] : 0.f, uhk = key < n ? suh[kk] : 0.f;
          const float E = __expf(S[r] * scale - M) * iZ;
          const float p = uk * E;
          const float pz = p * Sh[r] * scale + uhk * E;
          const float aj = sa[kk], bj = sb[kk];
          am += p * aj;
          bm += p * bj;
          zm += pz;
          pbz += pz * bj;
        }
      }
      am = sum_j4(am);
      bm = sum_j4(bm);
      zm = sum_j4(zm);
      pbz = sum_j4(pbz);
      const float ue = su[qc], uh = suh[qc];
      const float SP = ue * (am + pbz - 2.f * zm * bm) + uh * bm;
      if (j4 == 0 && qq < n) {
        bm_[qq] = bm;
        zm_[qq] = zm;
        sp_[qq] = SP;
        lq_[qq] = ue * (am + pbz - zm * bm) + uh * bm;   // query part of the adjoint of log u
      }
      f32x4v QB[OT];
#pragma unroll
      for (int t = 0; t < OT; ++t) QB[t] = zero4();
      for (int kt = 0; kt < nt; ++kt) {
        float kf[CG], khf[CG];
        fragw<CG>(QKV, ld, e0, n, kt * 16 + i16, ck + CG * j4, kf);
        fragw<CG>(QKVh, ld, e0, n, kt * 16 + i16, ck + CG * j4, khf);
        const f32x4v S = score_kq<CG>(kf, qf, zero4());
        const f32x4v Sh = score_kq<CG>(khf, qf, score_kq<CG>(kf, qhf, zero4()));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int key = kt * 16 + 4 * j4 + r;
          const int kk = key < n ? key : n - 1;
          const float uk = key < n ? su[kk] : 0.f, uhk = key < n ? suh[kk] : 0.f;
          const float E = __expf(S[r] * scale - M) * iZ;
          const float p = uk * E;
          const float pz = p * Sh[r] * scale + uhk * E;
          const float aj = sa[kk], bj = sb[kk];
          const float zb = ue * (p * aj + bj * (pz - p * zm) - pz * bm) + uh * p * bj - p * SP;
          const float zhb = ue * p * (bj - bm);
          float kc[OT], hc[OT];
          colsw<OT>(QKV, ld, e0, n, key, ck, i16, kc);
          colsw<OT>(QKVh, ld, e0, n, key, ck, i16, hc);
#pragma unroll
          for (int t = 0; t < OT; ++t) QB[t] = mfma16(zb, kc[t], QB[t]);
#pragma unroll
          for (int t = 0; t < OT; ++t) QB[t] = mfma16(zhb, hc[t], QB[t]);
        }
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int q = qt * 16 + 4 * j4 + r;
        if (q < n) {
          float* out = QKVa + (long long)(e0 + q) * ld + cq + i16;
#pragma unroll
          for (int t = 0; t < OT; ++t) out[16 * t] = QB[t][r] * scale;
        }
      }
    }
    wave_sync();
    // keys: kb and vb
    float alc[OT], bec[OT];
#pragma unroll
    for (int t = 0; t < OT; ++t) {
      alc[t] = al[16 * t + i16];
      bec[t] = be[16 * t + i16];
    }
    for (int kt = 0; kt < nt; ++kt) {
      float kf[CG], khf[CG];
      fragw<CG>(QKV, ld, e0, n, kt * 16 + i16, ck + CG * j4, kf);
      fragw<CG>(QKVh, ld, e0, n, kt * 16 + i16, ck + CG * j4, khf);
      const int kn = kt * 16 + i16, kc = kn < n ? kn : n - 1;
      const float uk = kn < n ? su[kc] : 0.f, uhk = kn < n ? suh[kc] : 0.f;
      const float aj = sa[kc], bj = sb[kc];
      f32x4v KB[OT];
#pragma unroll
      for (int t = 0; t < OT; ++t) KB[t] = zero4();
      float S1 = 0.f, S2 = 0.f, Lk = 0.f;
      for (int qt = 0; qt < nt; ++qt) {
        float qf[CG], qhf[CG];
        fragw<CG>(QKV, ld, e0, n, qt * 16 + i16, cq + CG * j4, qf);
        fragw<CG>(QKVh, ld, e0, n, qt * 16 + i16, cq + CG * j4, qhf);
        const f32x4v S = score_qk<CG>(qf, kf, zero4());
        const f32x4v Sh = score_qk<CG>(qf, khf, score_qk<CG>(qhf, kf, zero4()));
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int q = qt * 16 + 4 * j4 + r;
          const int qc = q < n ? q : n - 1;
          // padded query rows take no part (p = pz = 0)
          const float E = q < n ? __expf(S[r] * scale - sM[qc]) * siZ[qc] : 0.f;
          const float p = uk * E;
          const float pz = p * Sh[r] * scale + uhk * E;
          const float ue = q < n ? su[qc] : 0.f, uh = q < n ? suh[qc] : 0.f;
          const float bm = bm_[qc], zm = zm_[qc], SP = sp_[qc];
          const float zb = ue * (p * aj + bj * (pz - p * zm) - pz * bm) + uh * p * bj - p * SP;
          const float zhb = ue * p * (bj - bm);
          S1 += ue * p;
          S2 += uh * p + ue * (pz - p * zm);
          Lk += zb;   // key part of the adjoint of log u: sum over queries of the score adjoint
          float qv[OT], hv[OT];
          colsw<OT>(QKV, ld, e0, n, q, cq, i16, qv);
          colsw<OT>(QKVh, ld, e0, n, q, cq, i16, hv);
#pragma unroll
          for (int t = 0; t < OT; ++t) KB[t] = mfma16(zb, qv[t], KB[t]);
#pragma unroll
          for (int t = 0; t < OT; ++t) KB[t] = mfma16(zhb, hv[t], KB[t]);
        }
      }
      S1 = sum_j4(S1);
      S2 = sum_j4(S2);
      if (rlh) {
        Lk = sum_j4(Lk);
        if (j4 == 0 && kn < n) rlh[(long long)(e0 + kn) * H + a] = Lk + lq_[kn];
      }
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const int key = kt * 16 + 4 * j4 + r;
        const float S1r = __shfl(S1, 4 * j4 + r, 64), S2r = __shfl(S2, 4 * j4 + r, 64);
        if (key < n) {
          float* out = QKVa + (long long)(e0 + key) * ld;
#pragma unroll
          for (int t = 0; t < OT; ++t) out[ck + 16 * t + i16] = KB[t][r] * scale;
#pragma unroll
          for (int t = 0; t < OT; ++t) out[cv + 16 * t + i16] = S1r * alc[t] + S2r * bec[t];
        }
      }
    }
  }
}

}  // namespace janus
