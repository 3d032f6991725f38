// Bond-triplet (three-body) kernels of the training step.
//
// Paper Sec. "MatRIS": pairs of bonds sharing an atom define bond angles that
// become angle features; each interaction block has a three-body operation.
// Reading (the one the whole build follows): a triplet tau = (e, e2) is an
// ordered pair of distinct edges out of one centre, both shorter than r3
// under the pinned fp32 test; its features are
//   G[l, n] = P_l(c) B3_n(r_e2) u3(r_e),   c = u_e . u_e2,
// its token Z = (G W_a) * h_{j(e2)} goes through a routed expert MLP, and the
// messages of the triplets of e are added to the edge token X_e.
//
// Triplets are stored in CSR order by their first edge e (tseg(e)); trev[tau]
// is the triplet (e2, e).  Sums over "triplets whose second edge is e2" walk
// tseg(e2) through trev, and sums over "triplets whose second edge points to
// atom a" then walk seg(a) through the edge reverse map, so no kernel needs
// atomics.
//
// Inside the kernels the product of the features with W_a never materialises
// G: with s_l[col] = sum_n B3_n W_a[l Nb + n, col] (and s'_l with B3'),
//   (G W_a)       = u3 sum_l P_l  s_l
//   (dG/dc W_a)   = u3 sum_l P'_l s_l
//   (dG/dr2 W_a)  = u3 sum_l P_l  s'_l
//   (dG/dr1 W_a)  = u3' sum_l P_l s_l .
// The sums over l are polynomials in c of degree < L whose coefficients depend
// on the second edge only: the expert-token kernels rewrite s_l and s'_l once per
// edge in powers of c (a_k = sum_l C_lk s_l, C_lk the coefficient of c^k in P_l)
// and evaluate each triplet's value and c-derivative by Horner's rule.
#pragma once

#include "edge.h"
#include "gemm.h"

namespace janus {

constexpr int kMaxL = 8;

// Waves per SIMD the per-triplet kernels are compiled for: four (128 registers) while
// a lane holds at most 2 columns of a row, two (256) for the wider rows of d = 256 and
// 512, whose sums and derivative rows do not fit 128 registers.  The force-backward
// kernel at d = 512 (8 columns per lane) runs one wave per SIMD: at two it spills, and
// took twice as long; the other two spill little or nothing at two and stay there.
template <int VPL>
constexpr int kTriWaves = VPL <= 2 ? 4 : 2;
template <int VPL>
constexpr int kTriWavesP2 = VPL <= 4 ? kTriWaves<VPL> : 1;

__device__ __forceinline__ void legendre_d(float c, int L, float* P, float* dP) {
  P[0] = 1.f;
  dP[0] = 0.f;
  if (L > 1) {
    P[1] = c;
    dP[1] = 1.f;
  }
  for (int l = 1; l + 1 < L; ++l) {
    P[l + 1] = ((2 * l + 1) * c * P[l] - l * P[l - 1]) / (l + 1);
    dP[l + 1] = (l + 1) * P[l] + c * dP[l];
  }
}

// ---------------------------------------------------------------- builder

// short[e] = 1 iff the pinned fp32 test holds with r3 (same expression as the
// neighbour list).
__global__ void tri_short_kernel(const float* __restrict__ pos, const float* __restrict__ cell,
                                 const int* __restrict__ sid, const int* __restrict__ ei, const int* __restrict__ ej,
                                 const int8_t* __restrict__ shift, long long Ne, float rc3,
                                 unsigned char* __restrict__ sh) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const int i = ei[e], j = ej[e];
  const float* L = cell + 9 * sid[i];
  const float fx = shift[3 * e], fy = shift[3 * e + 1], fz = shift[3 * e + 2];
  const float sx = __fadd_rn(__fadd_rn(__fmul_rn(fx, L[0]), __fmul_rn(fy, L[3])), __fmul_rn(fz, L[6]));
  const float sy = __fadd_rn(__fadd_rn(__fmul_rn(fx, L[1]), __fmul_rn(fy, L[4])), __fmul_rn(fz, L[7]));
  const float sz = __fadd_rn(__fadd_rn(__fmul_rn(fx, L[2]), __fmul_rn(fy, L[5])), __fmul_rn(fz, L[8]));
  const float dx = __fadd_rn(__fsub_rn(pos[3 * j], pos[3 * i]), sx);
  const float dy = __fadd_rn(__fsub_rn(pos[3 * j + 1], pos[3 * i + 1]), sy);
  const float dz = __fadd_rn(__fsub_rn(pos[3 * j + 2], pos[3 * i + 2]), sz);
  const float r2 = __fadd_rn(__fadd_rn(__fmul_rn(dx, dx), __fmul_rn(dy, dy)), __fmul_rn(dz, dz));
  sh[e] = r2 < __fmul_rn(rc3, rc3) ? 1 : 0;
}

// Triplets of each edge: n_short(i) - 1 when e is short, else 0.
__global__ void tri_count_kernel(const int* __restrict__ rowptr, const unsigned char* __restrict__ sh, int N,
                                 int* __restrict__ tcount) {
  const int a = blockIdx.x * blockDim.x + threadIdx.x;
  if (a >= N) return;
  int ns = 0;
  for (int e = rowptr[a]; e < rowptr[a + 1]; ++e) ns += sh[e];
  for (int e = rowptr[a]; e < rowptr[a + 1]; ++e) tcount[e] = sh[e] ? ns - 1 : 0;
}

// Triplets per structure: sum over its atoms of ns (ns - 1).
__global__ void tri_struct_count_kernel(const int* __restrict__ offsets, const int* __restrict__ rowptr,
                                        const unsigned char* __restrict__ sh, int S, long long* __restrict__ out) {
  JANUS_WAVE_LOOP(s, S) {
    long long acc = 0;
    for (int a = offsets[s] + l; a < offsets[s + 1]; a += 64) {
      int ns = 0;
      for (int e = rowptr[a]; e < rowptr[a + 1]; ++e) ns += sh[e];
      acc += (long long)ns * (ns - 1);
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (l == 0) out[s] = acc;
  }
}

__global__ void tri_write_kernel(const int* __restrict__ ei, const int* __restrict__ rowptr,
                                 const unsigned char* __restrict__ sh, const int* __restrict__ trowptr, long long Ne,
                                 int* __restrict__ te, int* __restrict__ te2) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne || !sh[e]) return;
  const int i = ei[e];
  int p = trowptr[e];
  for (int f = rowptr[i]; f < rowptr[i + 1]; ++f)
    if (sh[f] && f != e) {
      te[p] = (int)e;
      te2[p] = f;
      ++p;
    }
}

// trev[tau] = index of (e2, e) in tseg(e2) (binary search on te2, which is
// increasing inside a segment); c[tau] = u_e . u_e2.
__global__ void tri_rev_kernel(const int* __restrict__ te, const int* __restrict__ te2,
                               const int* __restrict__ trowptr, const float4* __restrict__ geo, long long Nt,
                               int* __restrict__ trev, float* __restrict__ tc) {
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Nt) return;
  const int e = te[t], e2 = te2[t];
  int lo = trowptr[e2], hi = trowptr[e2 + 1];
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (te2[mid] < e) lo = mid + 1; else hi = mid;
  }
  trev[t] = (lo < trowptr[e2 + 1] && te2[lo] == e) ? lo : (int)t;
  const float4 a = geo[e], b = geo[e2];
  tc[t] = a.x * b.x + a.y * b.y + a.z * b.z;
}

// ---------------------------------------------------------------- routing

// Per triplet: logits ((P3a[Z_i] + P3b[Z_j(e)]) + P3c[Z_j(e2)]) + beta3 in
// fp32 for the top-k decision (lower index first on ties), gates from the
// float64 softmax.
__global__ void tri_route_kernel(const int* __restrict__ species, const int* __restrict__ ei,
                                 const int* __restrict__ ej, const int* __restrict__ te, const int* __restrict__ te2,
                                 long long Nt, const float* __restrict__ Pa, const float* __restrict__ Pb,
                                 const float* __restrict__ Pc, const float* __restrict__ beta, int E, int k,
                                 int* __restrict__ eid, float* __restrict__ gate) {
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Nt) return;
  const int za = species[ei[te[t]]], zb = species[ej[te[t]]], zc = species[ej[te2[t]]];
  float l[64];
  double mx = -1e300;
  for (int x = 0; x < E; ++x) {
    const float a = Pa[za * E + x], b = Pb[zb * E + x], c = Pc[zc * E + x], bt = beta[x];
    l[x] = __fadd_rn(__fadd_rn(__fadd_rn(a, b), c), bt);
    const double ld = (((double)a + (double)b) + (double)c) + (double)bt;
    mx = ld > mx ? ld : mx;
  }
  double den = 0.0;
  for (int x = 0; x < E; ++x)
    den += exp(((((double)Pa[za * E + x] + (double)Pb[zb * E + x]) + (double)Pc[zc * E + x]) + (double)beta[x]) - mx);
  unsigned long long taken = 0;
  for (int c = 0; c < k; ++c) {
    int best = -1;
    for (int x = 0; x < E; ++x) {
      if (taken >> x & 1ull) continue;
      if (best < 0 || l[x] > l[best]) best = x;
    }
    taken |= 1ull << best;
    eid[t * k + c] = best;
    gate[t * k + c] = (float)(exp(((((double)Pa[za * E + best] + (double)Pb[zb * E + best]) +
                                    (double)Pc[zc * E + best]) + (double)beta[best]) - mx) / den);
  }
}

// ---------------------------------------------------------------- feature rows
//
// The expert-token kernels run one wave per second edge e2: the sums
//   s_l = sum_n B3_n(r_e2) W_a[l Nb + n, :]   (and s'_l with B3')
// depend on e2 only, so they are formed once per edge; each triplet
// tau = (e, e2) then needs only its cosine c_tau and u3(r_e).
// The triplets whose second edge is e2 are trev[tseg(e2)]; their indices,
// cosines, u3 values and slot positions, stored once per step (per block for
// the slots) in that order, are loaded one triplet per lane, 64 at a time, and
// broadcast with readlane.

// Power-series coefficients of the Legendre polynomials, C[l][k] = [c^k] P_l(c),
// from Bonnet's recursion (l + 1) P_{l+1} = (2 l + 1) c P_l - l P_{l-1}.
struct LegendreCoef {
  float c[kMaxL][kMaxL];
};
constexpr LegendreCoef legendre_coef() {
  double t[kMaxL][kMaxL] = {};
  t[0][0] = 1.0;
  t[1][1] = 1.0;
  for (int l = 1; l + 1 < kMaxL; ++l)
    for (int k = 0; k < kMaxL; ++k)
      t[l + 1][k] = ((2 * l + 1) * (k > 0 ? t[l][k - 1] : 0.0) - l * t[l - 1][k]) / (l + 1);
  LegendreCoef m{};
  for (int l = 0; l < kMaxL; ++l)
    for (int k = 0; k < kMaxL; ++k) m.c[l][k] = (float)t[l][k];
  return m;
}
constexpr LegendreCoef kLegendreCoef = legendre_coef();

// s[l] (Legendre basis, zero for l >= L) -> a[k] = sum_l C[l][k] s[l] (powers of c).
template <int VPL>
__device__ __forceinline__ void legendre_to_powers(float (&s)[kMaxL][VPL]) {
  float a[kMaxL][VPL];
#pragma unroll
  for (int k = 0; k < kMaxL; ++k) {
#pragma unroll
    for (int v = 0; v < VPL; ++v) a[k][v] = 0.f;
#pragma unroll
    for (int l = k; l < kMaxL; ++l) {
      if (kLegendreCoef.c[l][k] != 0.f) {
#pragma unroll
        for (int v = 0; v < VPL; ++v) a[k][v] += kLegendreCoef.c[l][k] * s[l][v];
      }
    }
  }
#pragma unroll
  for (int k = 0; k < kMaxL; ++k)
#pragma unroll
    for (int v = 0; v < VPL; ++v) s[k][v] = a[k][v];
}

__device__ __forceinline__ float bcast(float x, int q) {
  return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), q));
}
__device__ __forceinline__ int bcast(int x, int q) { return __builtin_amdgcn_readlane(x, q); }

// s[q] = sum_n b_n sWa[(q Nb + n), cols of lane l] for q < L (b held one value per
// lane), returned in powers of c.
template <int VPL>
__device__ __forceinline__ void feat_sums(float b_lane, const float* sWa, int nb, int L, int d, int l,
                                          float (&s)[kMaxL][VPL]) {
#pragma unroll
  for (int q = 0; q < kMaxL; ++q) zero_row<VPL>(s[q]);
  for (int n = 0; n < nb; ++n) {
    const float b = bcast(b_lane, n);
#pragma unroll
    for (int q = 0; q < kMaxL; ++q) {
      if (q < L) {
        float w[VPL];
        ld_row<VPL>(sWa + (q * nb + n) * d, l, w);
#pragma unroll
        for (int v = 0; v < VPL; ++v) s[q][v] += b * w[v];
      }
    }
  }
  legendre_to_powers<VPL>(s);
}

// The same sums for two basis rows (B3 and B3') in one pass over W_a.
template <int VPL>
__device__ __forceinline__ void feat_sums2(float b_lane, float db_lane, const float* sWa, int nb, int L, int d, int l,
                                           float (&s)[kMaxL][VPL], float (&sp)[kMaxL][VPL]) {
#pragma unroll
  for (int q = 0; q < kMaxL; ++q) {
    zero_row<VPL>(s[q]);
    zero_row<VPL>(sp[q]);
  }
  for (int n = 0; n < nb; ++n) {
    const float b = bcast(b_lane, n), db = bcast(db_lane, n);
#pragma unroll
    for (int q = 0; q < kMaxL; ++q) {
      if (q < L) {
        float w[VPL];
        ld_row<VPL>(sWa + (q * nb + n) * d, l, w);
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          s[q][v] += b * w[v];
          sp[q][v] += db * w[v];
        }
      }
    }
  }
  legendre_to_powers<VPL>(s);
  legendre_to_powers<VPL>(sp);
}

// Per-triplet scalars in second-edge order, once per step: position t' of trev
// holds (c, u3(r_e), u3'(r_e), tau as int bits) of triplet tau = trev[t'] = (e, e2),
// so the expert-token kernels read a batch of triplets with one coalesced load
// instead of three dependent gathers (trev, then tc and te, then u3).
__global__ void tri_lane_kernel(const int* __restrict__ trev, const int* __restrict__ te,
                                const float* __restrict__ tc, const float* __restrict__ u3,
                                const float* __restrict__ du3, long long Nt, float4* __restrict__ tlane) {
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Nt) return;
  const int tau = trev[t];
  const int e1 = te[tau];
  tlane[t] = make_float4(tc[tau], u3[e1], du3[e1], __int_as_float(tau));
}

// Slot positions of one block's triplet routing in the same order:
// pos3r[t' KC + k] = pos3[trev[t'] KC + k].
__global__ void tri_pos_rev_kernel(const int* __restrict__ trev, const int* __restrict__ pos3, long long Nt, int KC,
                                   int* __restrict__ pos3r) {
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Nt) return;
  const long long tau = trev[t];
  for (int k = 0; k < KC; ++k) pos3r[t * KC + k] = pos3[tau * KC + k];
}

// Per-triplet scalars of up to 64 triplets at positions tb + lane (< t1) of the
// second-edge order, one triplet per lane (lanes past t1 repeat the last triplet).
template <int KC>
struct TriLane {
  int tau;
  float c, u, du;
  int pos[KC];
  __device__ __forceinline__ void load(const float4* __restrict__ tlane, const int* __restrict__ pos3r, int tb,
                                       int t1, int l) {
    const int tl = tb + l < t1 ? tb + l : t1 - 1;
    const float4 v = tlane[tl];
    c = v.x;
    u = v.y;
    du = v.z;
    tau = __float_as_int(v.w);
#pragma unroll
    for (int k = 0; k < KC; ++k) pos[k] = pos3r[(long long)tl * KC + k];
  }
};

// Raw slot rows of the two triplets of a pass starting at q0 (indices clamped
// to n - 1, so a pass past the end re-reads valid rows and is never used).
template <int VPL, int KC>
struct PassRows {
  float r[2][KC][VPL];
  __device__ __forceinline__ void load(const float* __restrict__ rows, const TriLane<KC>& tl, int q0, int n, int d,
                                       int l) {
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const int q = q0 + x < n ? q0 + x : n - 1;
#pragma unroll
      for (int k = 0; k < KC; ++k) ld_row<VPL>(rows + (long long)bcast(tl.pos[k], q) * d, l, r[x][k]);
    }
  }
  __device__ __forceinline__ void sum(int x, float (&y)[VPL]) const {
    zero_row<VPL>(y);
#pragma unroll
    for (int k = 0; k < KC; ++k) add_row<VPL>(y, r[x][k]);
  }
};

// Rows of a per-triplet array (row = triplet index) for the two triplets of a pass.
template <int VPL, int KC>
struct PassTri {
  float r[2][VPL];
  __device__ __forceinline__ void load(const float* __restrict__ rows, const TriLane<KC>& tl, int q0, int n, int d,
                                       int l) {
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      const int q = q0 + x < n ? q0 + x : n - 1;
      ld_row<VPL>(rows + (long long)bcast(tl.tau, q) * d, l, r[x]);
    }
  }
};

// (G W_a) row of one triplet and, with DERIV, (dG/dc W_a), (dG/dr1 W_a), (dG/dr2 W_a),
// from the per-edge coefficients in powers of c (s, and sp for the B3' sums): value and
// c-derivative by one Horner pass over the kMaxL coefficients (those of degree >= L
// are zero).
template <int VPL, bool DERIV>
__device__ __forceinline__ void tri_feat(float c, float u, float du, int L, const float (&s)[kMaxL][VPL],
                                         const float (&sp)[kMaxL][VPL], float (&z)[VPL], float (&wc)[VPL],
                                         float (&w1)[VPL], float (&w2)[VPL]) {
  (void)L;
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    z[v] = s[kMaxL - 1][v];
    if (DERIV) {
      wc[v] = 0.f;
      w2[v] = sp[kMaxL - 1][v];
    }
  }
#pragma unroll
  for (int k = kMaxL - 2; k >= 0; --k)
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      if (DERIV) {
        wc[v] = wc[v] * c + z[v];
        w2[v] = w2[v] * c + sp[k][v];
      }
      z[v] = z[v] * c + s[k][v];
    }
#pragma unroll
  for (int v = 0; v < VPL; ++v) {
    if (DERIV) {
      w1[v] = du * z[v];
      wc[v] *= u;
      w2[v] *= u;
    }
    z[v] *= u;
  }
}

// ---------------------------------------------------------------- phase 1

// Z_tau = (G W_a) * h_{j(e2)} into the triplet expert slots.
template <int VPL, int KC>
__global__ void tri_dispatch_kernel(const int* __restrict__ trowptr, const float4* __restrict__ tlane,
                                    const float* __restrict__ B3, const float* __restrict__ Wa, int nb, int L,
                                    const int* __restrict__ ej, const float* __restrict__ h,
                                    const int* __restrict__ pos3r, long long Ne, int d, float* __restrict__ Zs) {
  extern __shared__ float sWa[];
  load_lds(sWa, Wa, L * nb * d);
  JANUS_WAVE_LOOP(e2, Ne) {
    const int t0 = trowptr[e2], t1 = trowptr[e2 + 1];
    if (t0 == t1) continue;
    float s[kMaxL][VPL], hj[VPL];
    feat_sums<VPL>(basis_lane(B3, e2, nb, l), sWa, nb, L, d, l, s);
    ld_row<VPL>(h + (long long)ej[e2] * d, l, hj);
    for (int tb = t0; tb < t1; tb += 64) {
      TriLane<KC> tl;
      tl.load(tlane, pos3r, tb, t1, l);
      const int n = t1 - tb < 64 ? t1 - tb : 64;
      for (int q = 0; q < n; ++q) {
        float z[VPL], wc[VPL], w1[VPL], w2[VPL];
        tri_feat<VPL, false>(bcast(tl.c, q), bcast(tl.u, q), 0.f, L, s, s, z, wc, w1, w2);
        float Z[VPL];
#pragma unroll
        for (int v = 0; v < VPL; ++v) Z[v] = z[v] * hj[v];
#pragma unroll
        for (int k = 0; k < KC; ++k) st_row<VPL>(Zs + (long long)bcast(tl.pos[k], q) * d, l, Z);
      }
    }
  }
}

// Q_e = sum_{tau in tseg(e)} sum_c Y3g[pos3[tau, c]]  (gated triplet messages).
template <int VPL, int KC>
__global__ void tri_combine_kernel(const int* __restrict__ trowptr, const int* __restrict__ pos3,
                                   const float* __restrict__ Yg, long long Ne, int d, float* __restrict__ Q) {
  JANUS_WAVE_LOOP(e, Ne) {
    float acc[VPL];
    zero_row<VPL>(acc);
    const int t0 = trowptr[e], t1 = trowptr[e + 1];
    int t = t0;
    // four triplets' slot rows in flight per step
    for (; t + 4 <= t1; t += 4) {
      float y[4][VPL];
#pragma unroll
      for (int u = 0; u < 4; ++u) sum_slots<VPL, KC>(Yg, pos3, t + u, d, l, y[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) add_row<VPL>(acc, y[u]);
    }
    for (; t < t1; ++t) {
      float y0[VPL];
      sum_slots<VPL, KC>(Yg, pos3, t, d, l, y0);
      add_row<VPL>(acc, y0);
    }
    st_row<VPL>(Q + e * d, l, acc);
  }
}

// Slot rows of an edge adjoint for the triplets of the edge:
// out[pos3[tau, c]] = (g3_tau,c) * src[e],  tau in tseg(e).
template <int VPL, int KC>
__global__ void tri_gather_kernel(const int* __restrict__ trowptr, const int* __restrict__ pos3,
                                  const float* __restrict__ gate3, const float* __restrict__ src, long long Ne, int d,
                                  float* __restrict__ out) {
  JANUS_WAVE_LOOP(e, Ne) {
    const int t0 = trowptr[e], t1 = trowptr[e + 1];
    if (t0 == t1) continue;
    float s[VPL];
    ld_row<VPL>(src + e * d, l, s);
    const long long f1 = (long long)t1 * KC;
    long long f = (long long)t0 * KC;
    // eight slot rows per step: their indices (and gates) are loaded together
    for (; f + 8 <= f1; f += 8) {
      int q[8];
      float g[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        q[u] = pos3[f + u];
        g[u] = gate3 ? gate3[f + u] : 1.f;
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float o[VPL];
#pragma unroll
        for (int v = 0; v < VPL; ++v) o[v] = g[u] * s[v];
        st_row<VPL>(out + (long long)q[u] * d, l, o);
      }
    }
    for (; f < f1; ++f) {
      const float g = gate3 ? gate3[f] : 1.f;
      float o[VPL];
#pragma unroll
      for (int v = 0; v < VPL; ++v) o[v] = g * s[v];
      st_row<VPL>(out + (long long)pos3[f] * d, l, o);
    }
  }
}

// ---------------------------------------------------------------- phase 2

// Per triplet tau = (e, e2): Zbar = sum_c Zbar_slot (kept); the feature-
// geometry adjoints acc[tau] += (Zbar * h_j2) . (dG/dc W_a, dG/dr1 W_a, dG/dr2 W_a);
// and P[e2] += sum over the triplets of e2 of Zbar * (G W_a) (routed to h_j2),
// added in trev[tseg(e2)] order.
template <int VPL, int KC>
__global__ __launch_bounds__(256, kTriWavesP2<VPL>) void tri_p2_kernel(const int* __restrict__ trowptr, const float4* __restrict__ tlane,
                              const float* __restrict__ B3, const float* __restrict__ dB3,
                              const float* __restrict__ Wa, int nb, int L, const int* __restrict__ ej,
                              const float* __restrict__ h, const int* __restrict__ pos3r, long long Ne, int d,
                              const float* __restrict__ Zbs, float* __restrict__ Zbar, float4* __restrict__ acc,
                              float* __restrict__ P) {
  extern __shared__ float sWa[];
  load_lds(sWa, Wa, L * nb * d);
  JANUS_WAVE_LOOP(e2, Ne) {
    const int t0 = trowptr[e2], t1 = trowptr[e2 + 1];
    if (t0 == t1) continue;
    float s[kMaxL][VPL], sp[kMaxL][VPL], hj[VPL], pr[VPL];
    feat_sums2<VPL>(basis_lane(B3, e2, nb, l), basis_lane(dB3, e2, nb, l), sWa, nb, L, d, l, s, sp);
    ld_row<VPL>(h + (long long)ej[e2] * d, l, hj);
    ld_row<VPL>(P + e2 * d, l, pr);
    for (int tb = t0; tb < t1; tb += 64) {
      TriLane<KC> tl;
      tl.load(tlane, pos3r, tb, t1, l);
      const int n = t1 - tb < 64 ? t1 - tb : 64;
      // lane q keeps the geometry adjoints of triplet q of the batch
      float my_ac = 0.f, my_a1 = 0.f, my_a2 = 0.f;
      // two triplets per pass, with the rows of the following pass loaded
      // before a pass is computed (buffers A and B alternate).  Every pass does
      // the same memory operations (a pass past the end repeats the last
      // triplet with identical stores and zero weight in the sums), so the
      // compiler's waits stay exact.
      auto pass = [&](const PassRows<VPL, KC>& cur, int q0) {
        float zb[2][VPL];
#pragma unroll
        for (int x = 0; x < 2; ++x) cur.sum(x, zb[x]);
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          const bool real = q0 + x < n;
          const int q = real ? q0 + x : n - 1;
          const float wgt = real ? 1.f : 0.f;
          const long long t = bcast(tl.tau, q);
          float z[VPL], wc[VPL], w1[VPL], w2[VPL];
          tri_feat<VPL, true>(bcast(tl.c, q), bcast(tl.u, q), bcast(tl.du, q), L, s, sp, z, wc, w1, w2);
          st_row<VPL>(Zbar + t * d, l, zb[x]);
          float ac = 0.f, a1 = 0.f, a2 = 0.f;
#pragma unroll
          for (int v = 0; v < VPL; ++v) {
            pr[v] += wgt * (zb[x][v] * z[v]);
            const float w = zb[x][v] * hj[v];
            ac += w * wc[v];
            a1 += w * w1[v];
            a2 += w * w2[v];
          }
          ac = wave_sum(ac);
          a1 = wave_sum(a1);
          a2 = wave_sum(a2);
          my_ac = l == q ? ac : my_ac;
          my_a1 = l == q ? a1 : my_a1;
          my_a2 = l == q ? a2 : my_a2;
        }
      };
      PassRows<VPL, KC> A, B;
      A.load(Zbs, tl, 0, n, d, l);
      for (int q0 = 0; q0 < n; q0 += 4) {
        B.load(Zbs, tl, q0 + 2, n, d, l);
        __builtin_amdgcn_sched_barrier(0);
        pass(A, q0);
        A.load(Zbs, tl, q0 + 4, n, d, l);
        __builtin_amdgcn_sched_barrier(0);
        pass(B, q0 + 2);
      }
      if (l < n) {
        const float4 g = acc[tl.tau];
        acc[tl.tau] = make_float4(g.x + my_ac, g.y + my_a1, g.z + my_a2, g.w);
      }
    }
    st_row<VPL>(P + e2 * d, l, pr);
  }
}

// Displacement adjoint of every edge from the triplet geometry adjoints
// (ac, a1, a2) of the triplets it belongs to:
//   first edge:  ac (u2 - c u1) / r1 + a1 u1;   second edge: ac (u1 - c u2) / r2 + a2 u2.
__global__ void tri_edge_vec_kernel(const int* __restrict__ trowptr, const int* __restrict__ trev,
                                    const int* __restrict__ te2, const float* __restrict__ tc,
                                    const float4* __restrict__ geo, const float4* __restrict__ acc, long long Ne,
                                    float4* __restrict__ gvec) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const float4 ue = geo[e];
  double gx = 0, gy = 0, gz = 0;
  for (int t = trowptr[e]; t < trowptr[e + 1]; ++t) {
    // tau = (e, e2): e is the first edge
    const float4 u2 = geo[te2[t]];
    const float c = tc[t];
    const float4 a = acc[t];
    const double f = a.x / ue.w;
    gx += f * (u2.x - c * ue.x) + a.y * ue.x;
    gy += f * (u2.y - c * ue.y) + a.y * ue.y;
    gz += f * (u2.z - c * ue.z) + a.y * ue.z;
    // tau' = (e2, e): e is the second edge
    const int tr = trev[t];
    const float cr = tc[tr];
    const float4 ar = acc[tr];
    const double fr = ar.x / ue.w;
    gx += fr * (u2.x - cr * ue.x) + ar.z * ue.x;
    gy += fr * (u2.y - cr * ue.y) + ar.z * ue.y;
    gz += fr * (u2.z - cr * ue.z) + ar.z * ue.z;
  }
  gvec[e] = make_float4((float)gx, (float)gy, (float)gz, 0.f);
}

// ---------------------------------------------------------------- phase 3

// Per triplet, once per step: the loss adjoints of the feature-geometry
// adjoints, ct = (ac~, a1~, a2~), from the displacement tangents Gt_e
// (phi_i(e) - phi_j(e), plus the strain term of the stress seeds):
//   ac~ = Gt_e . (u2 - c u1) / r1 + Gt_e2 . (u1 - c u2) / r2,  a1~ = rt_e,  a2~ = rt_e2.
__global__ void tri_ctilde_kernel(const int* __restrict__ te, const int* __restrict__ te2,
                                  const float* __restrict__ tc, const float4* __restrict__ geo,
                                  const float4* __restrict__ gt, const float* __restrict__ rt, long long Nt,
                                  float4* __restrict__ ct) {
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Nt) return;
  const int e = te[t], e2 = te2[t];
  const float4 u1 = geo[e], u2 = geo[e2];
  const float c = tc[t];
  const float4 G1 = gt[e], G2 = gt[e2];
  const float g1x = G1.x, g1y = G1.y, g1z = G1.z;
  const float g2x = G2.x, g2y = G2.y, g2z = G2.z;
  const float acx = (g1x * (u2.x - c * u1.x) + g1y * (u2.y - c * u1.y) + g1z * (u2.z - c * u1.z)) / u1.w +
                    (g2x * (u1.x - c * u2.x) + g2y * (u1.y - c * u2.y) + g2z * (u1.z - c * u2.z)) / u2.w;
  ct[t] = make_float4(acx, rt[e], rt[e2], 0.f);
}

// Double backward per triplet tau = (e, e2) (Q = loss adjoint of hbar^t at
// j(e2), may be null):
//   vt   = ct . (dG W_a)            (adjoint of Zbar * h_j2)
//   Zbt  = vt * h_j2 + Q * (G W_a)  -> slots of the triplet
//   V    = Zbar * h_j2              (dW_a += Gt^T V)
// and P[e2] = sum over the triplets of e2 of vt * Zbar (routed to h_j2),
// written for every edge (zero without triplets).
template <int VPL, int KC>
__global__ __launch_bounds__(256, kTriWaves<VPL>) void tri_p3_kernel(const int* __restrict__ trowptr, const float4* __restrict__ tlane,
                              const float* __restrict__ B3, const float* __restrict__ dB3,
                              const float* __restrict__ Wa, int nb, int L, const int* __restrict__ ej,
                              const float* __restrict__ h, const float* __restrict__ hht,
                              const float4* __restrict__ ct, const float* __restrict__ Zbar,
                              const int* __restrict__ pos3r, long long Ne, int d, float* __restrict__ Zbts,
                              float* __restrict__ V, float* __restrict__ P) {
  extern __shared__ float sWa[];
  load_lds(sWa, Wa, L * nb * d);
  JANUS_WAVE_LOOP(e2, Ne) {
    const int t0 = trowptr[e2], t1 = trowptr[e2 + 1];
    float pr[VPL];
    zero_row<VPL>(pr);
    if (t0 < t1) {
      float s[kMaxL][VPL], sp[kMaxL][VPL], hj[VPL], qh[VPL];
      feat_sums2<VPL>(basis_lane(B3, e2, nb, l), basis_lane(dB3, e2, nb, l), sWa, nb, L, d, l, s, sp);
      const long long j2 = ej[e2];
      ld_row<VPL>(h + j2 * d, l, hj);
      if (hht) ld_row<VPL>(hht + j2 * d, l, qh); else zero_row<VPL>(qh);
      for (int tb = t0; tb < t1; tb += 64) {
        TriLane<KC> tl;
        tl.load(tlane, pos3r, tb, t1, l);
        const float4 cl = ct[tl.tau];
        const int n = t1 - tb < 64 ? t1 - tb : 64;
        auto pass = [&](const PassTri<VPL, KC>& cur, int q0) {
#pragma unroll
          for (int x = 0; x < 2; ++x) {
            const bool real = q0 + x < n;
            const int q = real ? q0 + x : n - 1;
            const float wgt = real ? 1.f : 0.f;
            const long long t = bcast(tl.tau, q);
            float z[VPL], wc[VPL], w1[VPL], w2[VPL];
            tri_feat<VPL, true>(bcast(tl.c, q), bcast(tl.u, q), bcast(tl.du, q), L, s, sp, z, wc, w1, w2);
            const float cx = bcast(cl.x, q), cy = bcast(cl.y, q), cz = bcast(cl.z, q);
            float Zb[VPL], vv[VPL];
#pragma unroll
            for (int v = 0; v < VPL; ++v) {
              const float vt = cx * wc[v] + cy * w1[v] + cz * w2[v];
              Zb[v] = vt * hj[v] + qh[v] * z[v];
              vv[v] = cur.r[x][v] * hj[v];
              pr[v] += wgt * (vt * cur.r[x][v]);
            }
            st_row<VPL>(V + t * d, l, vv);
#pragma unroll
            for (int k = 0; k < KC; ++k) st_row<VPL>(Zbts + (long long)bcast(tl.pos[k], q) * d, l, Zb);
          }
        };
        PassTri<VPL, KC> A, B;
        A.load(Zbar, tl, 0, n, d, l);
        for (int q0 = 0; q0 < n; q0 += 4) {
          B.load(Zbar, tl, q0 + 2, n, d, l);
          __builtin_amdgcn_sched_barrier(0);
          pass(A, q0);
          A.load(Zbar, tl, q0 + 4, n, d, l);
          __builtin_amdgcn_sched_barrier(0);
          pass(B, q0 + 2);
        }
      }
    }
    st_row<VPL>(P + e2 * d, l, pr);
  }
}

// Per edge, double backward of the triplet gather: gate adjoints
// g3t[tau, c] = Ybt3[pos3] . Xbar_e and QX_e = sum_tau sum_c g3 Ybt3[pos3].
template <int VPL, int KC>
__global__ void tri_combine_p3_kernel(const int* __restrict__ trowptr, const int* __restrict__ pos3,
                                      const float* __restrict__ gate3, const float* __restrict__ Ybt3,
                                      const float* __restrict__ Xbar, long long Ne, int d, float* __restrict__ g3t,
                                      float* __restrict__ QX) {
  JANUS_WAVE_LOOP(e, Ne) {
    float xb[VPL], acc[VPL];
    ld_row<VPL>(Xbar + e * d, l, xb);
    zero_row<VPL>(acc);
    const long long f1 = (long long)trowptr[e + 1] * KC;
    long long f = (long long)trowptr[e] * KC;
    // eight slot rows in flight per step; each row's dot product with Xbar goes
    // to lane u of the g3t store
    for (; f + 8 <= f1; f += 8) {
      float y[8][VPL], g[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        ld_row<VPL>(Ybt3 + (long long)pos3[f + u] * d, l, y[u]);
        g[u] = gate3[f + u];
      }
      float o = 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float su = 0.f;
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          su += y[u][v] * xb[v];
          acc[v] += g[u] * y[u][v];
        }
        su = wave_sum(su);
        o = l == u ? su : o;
      }
      if (l < 8) g3t[f + l] = o;
    }
    for (; f < f1; ++f) {
      float y[VPL];
      ld_row<VPL>(Ybt3 + (long long)pos3[f] * d, l, y);
      const float g = gate3[f];
      float su = 0.f;
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        su += y[v] * xb[v];
        acc[v] += g * y[v];
      }
      su = wave_sum(su);
      if (l == 0) g3t[f] = su;
    }
    st_row<VPL>(QX + e * d, l, acc);
  }
}

// ---------------------------------------------------------------- phase 4

// Per triplet tau = (e, e2), final backward: Zt = sum_c Zt_slot;
//   ZP = Zt * h_j2 + Q * Zbar   (loss adjoint of G W_a; dW_a += G^T ZP)
// and P[e2] += sum over the triplets of e2 of Zt * (G W_a) (routed to h_j2).
template <int VPL, int KC>
__global__ __launch_bounds__(256, kTriWaves<VPL>) void tri_p4_kernel(const int* __restrict__ trowptr, const float4* __restrict__ tlane,
                              const float* __restrict__ B3, const float* __restrict__ Wa, int nb, int L,
                              const int* __restrict__ ej, const float* __restrict__ h,
                              const float* __restrict__ hht, const float* __restrict__ Zbar,
                              const int* __restrict__ pos3r, long long Ne, int d,
                              const float* __restrict__ Zts, float* __restrict__ ZP, float* __restrict__ P) {
  extern __shared__ float sWa[];
  load_lds(sWa, Wa, L * nb * d);
  JANUS_WAVE_LOOP(e2, Ne) {
    const int t0 = trowptr[e2], t1 = trowptr[e2 + 1];
    if (t0 == t1) continue;
    float s[kMaxL][VPL], hj[VPL], qh[VPL], pr[VPL];
    feat_sums<VPL>(basis_lane(B3, e2, nb, l), sWa, nb, L, d, l, s);
    const long long j2 = ej[e2];
    ld_row<VPL>(h + j2 * d, l, hj);
    if (hht) ld_row<VPL>(hht + j2 * d, l, qh); else zero_row<VPL>(qh);
    ld_row<VPL>(P + e2 * d, l, pr);
    for (int tb = t0; tb < t1; tb += 64) {
      TriLane<KC> tl;
      tl.load(tlane, pos3r, tb, t1, l);
      const int n = t1 - tb < 64 ? t1 - tb : 64;
      auto pass = [&](const PassRows<VPL, KC>& cur, const PassTri<VPL, KC>& curb, int q0) {
        float zt[2][VPL];
#pragma unroll
        for (int x = 0; x < 2; ++x) cur.sum(x, zt[x]);
#pragma unroll
        for (int x = 0; x < 2; ++x) {
          const bool real = q0 + x < n;
          const int q = real ? q0 + x : n - 1;
          const float wgt = real ? 1.f : 0.f;
          const long long t = bcast(tl.tau, q);
          float z[VPL], wc[VPL], w1[VPL], w2[VPL];
          tri_feat<VPL, false>(bcast(tl.c, q), bcast(tl.u, q), 0.f, L, s, s, z, wc, w1, w2);
          float zp[VPL];
#pragma unroll
          for (int v = 0; v < VPL; ++v) {
            zp[v] = zt[x][v] * hj[v] + qh[v] * curb.r[x][v];
            pr[v] += wgt * (zt[x][v] * z[v]);
          }
          st_row<VPL>(ZP + t * d, l, zp);
        }
      };
      PassRows<VPL, KC> A, B;
      PassTri<VPL, KC> Ab, Bb;
      A.load(Zts, tl, 0, n, d, l);
      Ab.load(Zbar, tl, 0, n, d, l);
      for (int q0 = 0; q0 < n; q0 += 4) {
        B.load(Zts, tl, q0 + 2, n, d, l);
        Bb.load(Zbar, tl, q0 + 2, n, d, l);
        __builtin_amdgcn_sched_barrier(0);
        pass(A, Ab, q0);
        A.load(Zts, tl, q0 + 4, n, d, l);
        Ab.load(Zbar, tl, q0 + 4, n, d, l);
        __builtin_amdgcn_sched_barrier(0);
        pass(B, Bb, q0 + 2);
      }
    }
    st_row<VPL>(P + e2 * d, l, pr);
  }
}

// Loss adjoint of the triplet router logits, one thread per triplet:
//   lt[t, x] = p[x] (pt[x] - sum_c p[eid_c] gt_c),  pt[x] = sum_c [eid_c = x] gt_c,
// p the float64 softmax of the triplet's logits.
__global__ void tri_logit_kernel(const int* __restrict__ species, const int* __restrict__ ei,
                                 const int* __restrict__ ej, const int* __restrict__ te, const int* __restrict__ te2,
                                 long long Nt, const float* __restrict__ Pa, const float* __restrict__ Pb,
                                 const float* __restrict__ Pc, const float* __restrict__ beta, int E, int k,
                                 const int* __restrict__ eid, const float* __restrict__ gt, float* __restrict__ lt) {
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Nt) return;
  const int za = species[ei[te[t]]], zb = species[ej[te[t]]], zc = species[ej[te2[t]]];
  auto logit = [&](int x) {
    return (((double)Pa[za * E + x] + (double)Pb[zb * E + x]) + (double)Pc[zc * E + x]) + (double)beta[x];
  };
  double mx = -1e300;
  for (int x = 0; x < E; ++x) mx = fmax(mx, logit(x));
  double den = 0.0;
  for (int x = 0; x < E; ++x) den += exp(logit(x) - mx);
  float s = 0.f;
  for (int c = 0; c < k; ++c) s += (float)(exp(logit(eid[t * k + c]) - mx) / den) * gt[t * k + c];
  for (int x = 0; x < E; ++x) {
    float pt = 0.f;
    for (int c = 0; c < k; ++c)
      if (eid[t * k + c] == x) pt += gt[t * k + c];
    const float p = (float)(exp(logit(x) - mx) / den);
    lt[t * E + x] = p * (pt - s);
  }
}

// Per edge e and expert x (one thread each): LB[e, x] = sum over tseg(e) of
// lt, LC[e, x] = sum over the triplets whose second edge is e.
__global__ void tri_router_edge_kernel(const int* __restrict__ trowptr, const int* __restrict__ trev, int E,
                                       const float* __restrict__ lt, long long Ne, float* __restrict__ LB,
                                       float* __restrict__ LC) {
  const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= Ne * E) return;
  const long long e = g / E;
  const int x = (int)(g - e * E);
  float b = 0.f, c = 0.f;
  for (int t = trowptr[e]; t < trowptr[e + 1]; ++t) {
    b += lt[(long long)t * E + x];
    c += lt[(long long)trev[t] * E + x];
  }
  LB[g] = b;
  LC[g] = c;
}

// Per atom: pa = sum over own edges of LB (vertex species), pb = sum over
// incoming edges of LB (species of j(e)), pc = sum over incoming edges of LC.
__global__ void tri_router_atom_kernel(const int* __restrict__ rowptr, const int* __restrict__ rev, int E,
                                       const float* __restrict__ LB, const float* __restrict__ LC, int N,
                                       float* __restrict__ pa, float* __restrict__ pb, float* __restrict__ pc) {
  JANUS_WAVE_LOOP(i, N) {
    float a = 0.f, b = 0.f, c = 0.f;
    if (l < E)
      for (int e = rowptr[i]; e < rowptr[i + 1]; ++e) {
        a += LB[(long long)e * E + l];
        b += LB[(long long)rev[e] * E + l];
        c += LC[(long long)rev[e] * E + l];
      }
    if (l < E) {
      pa[i * E + l] = a;
      pb[i * E + l] = b;
      pc[i * E + l] = c;
    }
  }
}

// ---------------------------------------------------------------- loaders

// Rows of the triplet features for weight-gradient products:
// plain: G[t, f]; with coefficients ct: ac~ dG/dc + a1~ dG/dr1 + a2~ dG/dr2.
struct LoadTriFeat {
  const int* te;
  const int* te2;
  const float* tc;
  const float* B3;
  const float* dB3;
  const float* u3;
  const float* du3;
  const float4* ct;   // null: plain features
  int nb;
  using Raw = float4;
  __device__ __forceinline__ Raw load(long long t, int f) const {
    const int q = f / nb, n = f - q * nb;
    float P[kMaxL], dP[kMaxL];
    legendre_d(tc[t], q + 1, P, dP);
    const int e1 = te[t], e2 = te2[t];
    const float4 b = ld4(B3 + (long long)e2 * nb + n);
    const float u = u3[e1];
    if (!ct) {
      const float s = P[q] * u;
      return make_float4(s * b.x, s * b.y, s * b.z, s * b.w);
    }
    const float4 db = ld4(dB3 + (long long)e2 * nb + n);
    const float4 cf = ct[t];
    const float du = du3[e1];
    const float kb = cf.x * dP[q] * u + cf.y * P[q] * du, kd = cf.z * P[q] * u;
    return make_float4(kb * b.x + kd * db.x, kb * b.y + kd * db.y, kb * b.z + kd * db.z, kb * b.w + kd * db.w);
  }
  __device__ __forceinline__ float4 apply(const Raw& v, int) const { return v; }
};

// Feature rows of every triplet, out[t, f] = ld.load(t, f), written once per
// step for the weight-gradient products of all blocks (the features do not
// depend on the block).  One thread per 4 consecutive features.
__global__ void tri_features_kernel(LoadTriFeat ld, long long Nt, int nf, float* __restrict__ out) {
  const int nq = nf / 4;
  const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= Nt * nq) return;
  const long long t = g / nq;
  const int f = 4 * (int)(g - t * nq);
  *reinterpret_cast<float4*>(out + t * nf + f) = ld.load(t, f);
}


// ---------------------------------------------------------- loss gradient in positions

// Loss gradient in the positions, bond-angle part, per triplet tau = (e, e2):
// with Ag = dL/dG_tau (the final backward's adjoint of the features) and
// Ad = -dE/dG-adjoint of the double backward (Ad = -sum_t W_a (Zbar * h_j2)),
// and the displacement tangents dd = -gt (gt_e = phi_i - phi_j + Psi_s d_e):
//   first partials:  (ac, a1, a2) = Ag . (dG/dc, dG/dr1, dG/dr2)
//     -> e:  ac (u2 - c u1) / r1 + a1 u1,   e2: ac (u1 - c u2) / r2 + a2 u2;
//   tangent part: the gradient in d_e, d_e2 of
//     s = Ad . (dG/dc cdot + dG/dr1 rdot1 + dG/dr2 rdot2),
//     rdot = dd . u,  udot = (dd - rdot u) / r,  cdot = udot1 . u2 + u1 . udot2,
//   which takes the second partials of G = P_l(c) B3_n(r2) u3(r1) (P'', B3'', u3'')
//   and, through dd = ... - Psi d, the stress seeds.
// Float64 throughout; one thread per triplet; the two vectors go to tp1 (for e)
// and tp2 (for e2).
__global__ __launch_bounds__(128, 2) void tri_pos_kernel(const int* __restrict__ te, const int* __restrict__ te2,
                               const float* __restrict__ tc, const float4* __restrict__ geo,
                               const float4* __restrict__ gt, const float* __restrict__ Psi,
                               const int* __restrict__ ei, const int* __restrict__ sid,
                               const float* __restrict__ Ag, const float* __restrict__ Adn, long long Nt, int nb,
                               int L, float r3f, float4* __restrict__ tp1, float4* __restrict__ tp2) {
  const long long t = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (t >= Nt) return;
  const int e1 = te[t], e2 = te2[t];
  const float4 g1 = geo[e1], g2 = geo[e2];
  const double u1[3] = {g1.x, g1.y, g1.z}, u2[3] = {g2.x, g2.y, g2.z};
  const double r1 = g1.w, r2 = g2.w, c = tc[t], r3 = r3f;
  const float4 q1 = gt[e1], q2 = gt[e2];
  const double dd1[3] = {-(double)q1.x, -(double)q1.y, -(double)q1.z};
  const double dd2[3] = {-(double)q2.x, -(double)q2.y, -(double)q2.z};
  const float* Ps = Psi ? Psi + 9 * sid[ei[e1]] : nullptr;
  // Legendre P, P', P'' at c (l < L): Bonnet's recursion and its derivatives
  double P[kMaxL], dP[kMaxL], d2P[kMaxL];
  P[0] = 1.0; dP[0] = 0.0; d2P[0] = 0.0;
  if (L > 1) { P[1] = c; dP[1] = 1.0; d2P[1] = 0.0; }
#pragma unroll
  for (int l = 1; l < kMaxL - 1; ++l) {
    if (l + 1 < L) {
      P[l + 1] = ((2 * l + 1) * c * P[l] - l * P[l - 1]) / (l + 1);
      dP[l + 1] = (l + 1) * P[l] + c * dP[l];
      d2P[l + 1] = (l + 2) * dP[l] + c * d2P[l];
    }
  }
  // envelope u3(r1) and its first two radial derivatives
  double e3 = 0.0, de3 = 0.0, d2e3 = 0.0;
  {
    const double x = r1 / r3;
    if (x < 1.0) {
      const double x2 = x * x, x4 = x2 * x2, x5 = x4 * x, x6 = x5 * x;
      e3 = 1.0 - 28.0 * x6 + 48.0 * x6 * x - 21.0 * x6 * x2;
      de3 = (-168.0 * x5 + 336.0 * x6 - 168.0 * x6 * x) / r3;
      d2e3 = (-840.0 * x4 + 2016.0 * x5 - 1176.0 * x6) / (r3 * r3);
    }
  }
  // B3_n(r2), B3_n', B3_n'' (n = 1..nb) summed against the two adjoints per l:
  //   SA[l] = sum_n Ad[l, n] B3_n, SA1 with B3', SA2 with B3''; SG, SG1 with Ag
  double SA[kMaxL], SA1[kMaxL], SA2[kMaxL], SG[kMaxL], SG1[kMaxL];
#pragma unroll
  for (int l = 0; l < kMaxL; ++l) SA[l] = SA1[l] = SA2[l] = SG[l] = SG1[l] = 0.0;
  {
    double u, du, d2u;
    const double x = r2 / r3;
    u = du = d2u = 0.0;
    if (x < 1.0) {
      const double x2 = x * x, x4 = x2 * x2, x5 = x4 * x, x6 = x5 * x;
      u = 1.0 - 28.0 * x6 + 48.0 * x6 * x - 21.0 * x6 * x2;
      du = (-168.0 * x5 + 336.0 * x6 - 168.0 * x6 * x) / r3;
      d2u = (-840.0 * x4 + 2016.0 * x5 - 1176.0 * x6) / (r3 * r3);
    }
    const double cn = sqrt(2.0 / r3), th = M_PI / r3, ir = 1.0 / r2;
    double s1, c1;
    sincos(th * r2, &s1, &c1);
    double sn = s1, cs = c1;
    const float* arow = Adn + t * (long long)(L * nb);
    const float* grow = Ag + t * (long long)(L * nb);
    for (int n = 0; n < nb; ++n) {
      const double k = (n + 1) * th;
      const double sr = sn * ir;
      const double ds = (k * cs - sr) * ir;
      const double d2s = -k * k * sr - 2.0 * ds * ir;
      const double b = cn * sr * u, db = cn * (ds * u + sr * du), d2b = cn * (d2s * u + 2.0 * ds * du + sr * d2u);
#pragma unroll
      for (int l = 0; l < kMaxL; ++l) {
        if (l < L) {
          const double a = -(double)arow[l * nb + n], g = grow[l * nb + n];
          SA[l] += a * b;
          SA1[l] += a * db;
          SA2[l] += a * d2b;
          SG[l] += g * b;
          SG1[l] += g * db;
        }
      }
      const double sn1 = sn * c1 + cs * s1;
      cs = cs * c1 - sn * s1;
      sn = sn1;
    }
  }
  double g_c = 0, g_1 = 0, g_2 = 0, g_cc = 0, g_c1 = 0, g_c2 = 0, g_11 = 0, g_12 = 0, g_22 = 0;
  double ac = 0, a1 = 0, a2 = 0;
#pragma unroll
  for (int l = 0; l < kMaxL; ++l) {
    if (l < L) {
      g_c += dP[l] * SA[l];
      g_1 += P[l] * SA[l];
      g_2 += P[l] * SA1[l];
      g_cc += d2P[l] * SA[l];
      g_c2 += dP[l] * SA1[l];
      g_22 += P[l] * SA2[l];
      ac += dP[l] * SG[l];
      a1 += P[l] * SG[l];
      a2 += P[l] * SG1[l];
    }
  }
  g_c1 = g_c * de3;   // <A, P' B3> u3'
  g_11 = g_1 * d2e3;  // <A, P B3> u3''
  g_12 = g_2 * de3;   // <A, P B3'> u3'
  g_c *= e3; g_1 *= de3; g_2 *= e3; g_cc *= e3; g_c2 *= e3; g_22 *= e3;
  ac *= e3; a1 *= de3; a2 *= e3;
  // Psi^T v of the triplet's structure (the tangent depends on d through -Psi d)
  auto PT = [&](const double (&v)[3], double (&o)[3]) {
    for (int k = 0; k < 3; ++k) o[k] = Ps ? (double)Ps[k] * v[0] + (double)Ps[3 + k] * v[1] + (double)Ps[6 + k] * v[2] : 0.0;
  };
  double rd1 = 0, rd2 = 0;
  for (int k = 0; k < 3; ++k) { rd1 += dd1[k] * u1[k]; rd2 += dd2[k] * u2[k]; }
  double ud1[3], ud2[3];
  for (int k = 0; k < 3; ++k) { ud1[k] = (dd1[k] - rd1 * u1[k]) / r1; ud2[k] = (dd2[k] - rd2 * u2[k]) / r2; }
  double w1 = 0, w2 = 0;
  for (int k = 0; k < 3; ++k) { w1 += ud1[k] * u2[k]; w2 += u1[k] * ud2[k]; }
  const double cd = w1 + w2;
  double pu1[3], pu2[3];
  PT(u1, pu1);
  PT(u2, pu2);
  const double a_c = g_cc * cd + g_c1 * rd1 + g_c2 * rd2;
  const double a_1 = g_c1 * cd + g_11 * rd1 + g_12 * rd2;
  const double a_2 = g_c2 * cd + g_12 * rd1 + g_22 * rd2;
  double o1[3], o2[3];
  for (int k = 0; k < 3; ++k) {
    const double gc1 = (u2[k] - c * u1[k]) / r1, gc2 = (u1[k] - c * u2[k]) / r2;
    const double grd1 = ud1[k] - pu1[k], grd2 = ud2[k] - pu2[k];
    const double gw1_d1 = (-pu2[k] - c * grd1 - rd1 * gc1 - w1 * u1[k]) / r1;
    const double gw2_d1 = (ud2[k] - w2 * u1[k]) / r1;
    const double gw2_d2 = (-pu1[k] - c * grd2 - rd2 * gc2 - w2 * u2[k]) / r2;
    const double gw1_d2 = (ud1[k] - w1 * u2[k]) / r2;
    o1[k] = a_c * gc1 + a_1 * u1[k] + g_c * (gw1_d1 + gw2_d1) + g_1 * grd1 + ac * gc1 + a1 * u1[k];
    o2[k] = a_c * gc2 + a_2 * u2[k] + g_c * (gw1_d2 + gw2_d2) + g_2 * grd2 + ac * gc2 + a2 * u2[k];
  }
  tp1[t] = make_float4((float)o1[0], (float)o1[1], (float)o1[2], 0.f);
  tp2[t] = make_float4((float)o2[0], (float)o2[1], (float)o2[2], 0.f);
}

// Per edge: the triplet vectors of the triplets where e is the first edge
// (tp1 over tseg(e)) and where it is the second (tp2 of trev over tseg(e)),
// added in triplet order.
__global__ void tri_pos_edge_kernel(const int* __restrict__ trowptr, const int* __restrict__ trev,
                                    const float4* __restrict__ tp1, const float4* __restrict__ tp2, long long Ne,
                                    float4* __restrict__ out) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  double x = 0, y = 0, z = 0;
  for (int t = trowptr[e]; t < trowptr[e + 1]; ++t) {
    const float4 a = tp1[t], b = tp2[trev[t]];
    x += (double)a.x + b.x;
    y += (double)a.y + b.y;
    z += (double)a.z + b.z;
  }
  out[e] = make_float4((float)x, (float)y, (float)z, 0.f);
}

}  // namespace janus
