// Edge- and atom-level kernels of the training step (wave64, one wave per
// edge or per atom).
//
// Notation (per interaction block t, edge e = (i, j, n), choice c):
//   F_e  = B(r_e) W_b          radial filter,   F'_e = B'(r_e) W_b
//   X_e  = F_e * h_j           edge token, copied into the slot pos[e, c] of
//                              each of its k experts
//   m_e  = sum_c g_ec Y_ec     gated expert outputs, summed into h_i
// Adjoints: a trailing "bar" is d(E_total)/d(.) of the force backward; the
// double backward and the final backward carry d(loss)/d(.) of those.
// Every sum over the edges of an atom walks its CSR segment in order; sums
// over the edges that point *to* an atom walk the segment through the
// reverse-edge map.  No kernel uses floating-point atomics.
//
// Memory access: the wave's item index is wave-uniform (readfirstlane), so
// per-item indices (pos, ej, rev, gates, segment bounds) are one address for
// the whole wave; a feature row of d = 64 VPL floats is read or written by the whole wave in
// VPL / W accesses of W = min(VPL, 4) consecutive floats per lane (Lanes),
// each covering one contiguous 256 W-byte segment.  The k slot rows of an
// edge (k is a template argument, 1..4) and, in the per-atom sums, the rows
// of two edges are loaded before any of them is used.
#pragma once

#include "common.h"

namespace janus {

constexpr int kMaxTopK = 4;

template <int VPL>
struct Lanes {
  static constexpr int W = VPL < 4 ? VPL : 4;   // floats per lane per access
  static constexpr int Q = VPL / W;             // accesses per row
  // column of x[q * W + w] for lane l: 64 W q + W l + w
  __device__ static __forceinline__ int col(int l, int q) { return 64 * W * q + W * l; }
};

template <int VPL>
__device__ __forceinline__ void ld_row(const float* __restrict__ p, int l, float (&x)[VPL]) {
  constexpr int W = Lanes<VPL>::W;
#pragma unroll
  for (int q = 0; q < Lanes<VPL>::Q; ++q) {
    const float* s = p + Lanes<VPL>::col(l, q);
    if constexpr (W == 4) {
      const float4 v = *reinterpret_cast<const float4*>(s);
      x[4 * q] = v.x; x[4 * q + 1] = v.y; x[4 * q + 2] = v.z; x[4 * q + 3] = v.w;
    } else if constexpr (W == 2) {
      const float2 v = *reinterpret_cast<const float2*>(s);
      x[2 * q] = v.x; x[2 * q + 1] = v.y;
    } else {
      x[q] = *s;
    }
  }
}

template <int VPL>
__device__ __forceinline__ void st_row(float* __restrict__ p, int l, const float (&x)[VPL]) {
  constexpr int W = Lanes<VPL>::W;
#pragma unroll
  for (int q = 0; q < Lanes<VPL>::Q; ++q) {
    float* s = p + Lanes<VPL>::col(l, q);
    if constexpr (W == 4) {
      *reinterpret_cast<float4*>(s) = make_float4(x[4 * q], x[4 * q + 1], x[4 * q + 2], x[4 * q + 3]);
    } else if constexpr (W == 2) {
      *reinterpret_cast<float2*>(s) = make_float2(x[2 * q], x[2 * q + 1]);
    } else {
      *s = x[q];
    }
  }
}

template <int VPL>
__device__ __forceinline__ void zero_row(float (&x)[VPL]) {
#pragma unroll
  for (int v = 0; v < VPL; ++v) x[v] = 0.f;
}

template <int VPL>
__device__ __forceinline__ void add_row(float (&x)[VPL], const float (&y)[VPL]) {
#pragma unroll
  for (int v = 0; v < VPL; ++v) x[v] += y[v];
}

// One basis row of an edge, one value per lane (lane n < nb holds b_n);
// nb <= 32, so a single coalesced load.
__device__ __forceinline__ float basis_lane(const float* __restrict__ B, long long e, int nb, int l) {
  return B[e * nb + (l < nb ? l : nb - 1)];
}

// F = b W_b for one edge, W_b [nb, d] staged in LDS; b is held one value per lane.
template <int VPL>
__device__ __forceinline__ void filter_row(float b_lane, const float* sW, int nb, int d, int l, float (&F)[VPL]) {
  zero_row<VPL>(F);
#pragma unroll 4
  for (int n = 0; n < nb; ++n) {
    const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(b_lane), n));
    float w[VPL];
    ld_row<VPL>(sW + n * d, l, w);
#pragma unroll
    for (int v = 0; v < VPL; ++v) F[v] += b * w[v];
  }
}

// F = b W_b and F' = b' W_b together: each staged row of W_b is read once.
template <int VPL>
__device__ __forceinline__ void filter_rows2(float b_lane, float db_lane, const float* sW, int nb, int d, int l,
                                             float (&F)[VPL], float (&Fp)[VPL]) {
  zero_row<VPL>(F);
  zero_row<VPL>(Fp);
#pragma unroll 4
  for (int n = 0; n < nb; ++n) {
    const float b = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(b_lane), n));
    const float db = __int_as_float(__builtin_amdgcn_readlane(__float_as_int(db_lane), n));
    float w[VPL];
    ld_row<VPL>(sW + n * d, l, w);
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      F[v] += b * w[v];
      Fp[v] += db * w[v];
    }
  }
}

__device__ __forceinline__ void load_lds(float* s, const float* g, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) s[i] = g[i];
  __syncthreads();
}

// Grid-stride loop of waves over items; the item index is wave-uniform.
#define JANUS_WAVE_LOOP(var, count)                                                                        \
  const int l = threadIdx.x & 63;                                                                          \
  const long long nw_ = (long long)gridDim.x * (blockDim.x >> 6);                                          \
  for (long long var = (long long)blockIdx.x * (blockDim.x >> 6) + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6); \
       var < (count); var += nw_)

// y = sum_c rows[pos[e, c]]  (the k slot rows of edge e)
template <int VPL, int KC>
__device__ __forceinline__ void sum_slots(const float* __restrict__ rows, const int* __restrict__ pos, long long e,
                                          int d, int l, float (&y)[VPL]) {
  float r[KC][VPL];
#pragma unroll
  for (int c = 0; c < KC; ++c) ld_row<VPL>(rows + (long long)pos[e * KC + c] * d, l, r[c]);
  zero_row<VPL>(y);
#pragma unroll
  for (int c = 0; c < KC; ++c) add_row<VPL>(y, r[c]);
}

// Phase 1: X_e = F_e * h_j (+ Q_e, the triplet messages of e when present),
// written to the slots of its k experts.
template <int VPL, int KC>
__global__ void dispatch_x_kernel(const float* __restrict__ B, int nb, const float* __restrict__ Wb,
                                  const float* __restrict__ h, const int* __restrict__ ej,
                                  const int* __restrict__ pos, long long Ne, int d, float* __restrict__ Xs,
                                  const float* __restrict__ Q) {
  extern __shared__ float sW[];
  load_lds(sW, Wb, nb * d);
  JANUS_WAVE_LOOP(e, Ne) {
    const float bl = basis_lane(B, e, nb, l);
    float hj[VPL], q[VPL];
    ld_row<VPL>(h + (long long)ej[e] * d, l, hj);
    if (Q) ld_row<VPL>(Q + e * d, l, q); else zero_row<VPL>(q);
    float F[VPL];
    filter_row<VPL>(bl, sW, nb, d, l, F);
    float X[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) X[v] = F[v] * hj[v] + q[v];
#pragma unroll
    for (int c = 0; c < KC; ++c) st_row<VPL>(Xs + (long long)pos[e * KC + c] * d, l, X);
  }
}

// Phase 1: h'_i = h_i + sum_{e in seg(i)} sum_c Yg[pos[e, c]]  (Yg already gated).
template <int VPL, int KC>
__global__ void combine_fwd_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos,
                                   const float* __restrict__ Yg, const float* __restrict__ h, int N, int d,
                                   float* __restrict__ hn) {
  JANUS_WAVE_LOOP(i, N) {
    float acc[VPL];
    ld_row<VPL>(h + i * d, l, acc);
    const int e0 = rowptr[i], e1 = rowptr[i + 1];
    int e = e0;
    // four edges' slot rows in flight per step (one wave per atom: the loop over the
    // neighbourhood is the wave's latency chain)
    for (; e + 4 <= e1; e += 4) {
      float y[4][VPL];
#pragma unroll
      for (int u = 0; u < 4; ++u) sum_slots<VPL, KC>(Yg, pos, e + u, d, l, y[u]);
#pragma unroll
      for (int u = 0; u < 4; ++u) add_row<VPL>(acc, y[u]);
    }
    for (; e < e1; ++e) {
      float y0[VPL];
      sum_slots<VPL, KC>(Yg, pos, e, d, l, y0);
      add_row<VPL>(acc, y0);
    }
    st_row<VPL>(hn + i * d, l, acc);
  }
}

// Slot rows of the adjoint arriving at the messages: out[pos[e, c]] = (g_ec) * src[i(e)].
template <int VPL, int KC>
__global__ void gather_atom_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos,
                                   const float* __restrict__ gate, const float* __restrict__ src, int N, int d,
                                   float* __restrict__ out) {
  JANUS_WAVE_LOOP(i, N) {
    float s[VPL];
    ld_row<VPL>(src + i * d, l, s);
    const long long f0 = (long long)rowptr[i] * KC, f1 = (long long)rowptr[i + 1] * KC;
    long long f = f0;
    // eight slot rows per step: their indices (and gates) are loaded together
    for (; f + 8 <= f1; f += 8) {
      int q[8];
      float g[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        q[u] = pos[f + u];
        g[u] = gate ? gate[f + u] : 1.f;
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
      const float g = gate ? gate[f] : 1.f;
      float o[VPL];
#pragma unroll
      for (int v = 0; v < VPL; ++v) o[v] = g * s[v];
      st_row<VPL>(out + (long long)pos[f] * d, l, o);
    }
  }
}

// Phase 2 per edge: Xbar_e = sum_c Xbar_slot (+ Xadd_e); Fbar = Xbar * h_j;
// rbar_e += Fbar . F'_e; P_e = Xbar * F_e (routed to h_j by scatter_rev).
template <int VPL, int KC>
__global__ void edge_p2_kernel(const float* __restrict__ B, const float* __restrict__ dB, int nb,
                               const float* __restrict__ Wb, const float* __restrict__ h, const int* __restrict__ ej,
                               const int* __restrict__ pos, long long Ne, int d, const float* __restrict__ Xbs,
                               float* __restrict__ Xbar, float* __restrict__ Fbar, float* __restrict__ rbar,
                               float* __restrict__ P, const float* __restrict__ Xadd) {
  extern __shared__ float sW[];
  load_lds(sW, Wb, nb * d);
  JANUS_WAVE_LOOP(e, Ne) {
    const float bl = basis_lane(B, e, nb, l), dbl = basis_lane(dB, e, nb, l);
    float xb[VPL], hj[VPL];
    sum_slots<VPL, KC>(Xbs, pos, e, d, l, xb);
    if (Xadd) {   // the router's part of Xbar (routing on the edge tokens)
      float xa[VPL];
      ld_row<VPL>(Xadd + e * d, l, xa);
      add_row<VPL>(xb, xa);
    }
    ld_row<VPL>(h + (long long)ej[e] * d, l, hj);
    float F[VPL], Fp[VPL];
    filter_rows2<VPL>(bl, dbl, sW, nb, d, l, F, Fp);
    float fb[VPL], p[VPL];
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      fb[v] = xb[v] * hj[v];
      p[v] = xb[v] * F[v];
      s += fb[v] * Fp[v];
    }
    st_row<VPL>(Xbar + e * d, l, xb);
    st_row<VPL>(Fbar + e * d, l, fb);
    st_row<VPL>(P + e * d, l, p);
    s = wave_sum(s);
    if (l == 0) rbar[e] += s;
  }
}

// out_a = base0_a (+ base1_a) + sum_{e' in seg(a)} P[rev(e')]: the sum over edges whose neighbour is a.
template <int VPL>
__global__ void scatter_rev_kernel(const int* __restrict__ rowptr, const int* __restrict__ rev,
                                   const float* __restrict__ P, const float* __restrict__ base0,
                                   const float* __restrict__ base1, int N, int d, float* __restrict__ out) {
  JANUS_WAVE_LOOP(a, N) {
    float acc[VPL];
    if (base0) ld_row<VPL>(base0 + a * d, l, acc); else zero_row<VPL>(acc);
    if (base1) {
      float b[VPL];
      ld_row<VPL>(base1 + a * d, l, b);
      add_row<VPL>(acc, b);
    }
    const int e0 = rowptr[a], e1 = rowptr[a + 1];
    int e = e0;
    // eight reverse edges' rows in flight per step
    for (; e + 8 <= e1; e += 8) {
      float pr[8][VPL];
#pragma unroll
      for (int u = 0; u < 8; ++u) ld_row<VPL>(P + (long long)rev[e + u] * d, l, pr[u]);
#pragma unroll
      for (int u = 0; u < 8; ++u) add_row<VPL>(acc, pr[u]);
    }
    for (; e < e1; ++e) {
      float p0[VPL];
      ld_row<VPL>(P + (long long)rev[e] * d, l, p0);
      add_row<VPL>(acc, p0);
    }
    st_row<VPL>(out + a * d, l, acc);
  }
}

// Phase 3 per edge (adjoints of the force backward):
//   Fbt = rt_e F'_e,  Xbt = Q_e * F_e + Fbt * h_j (+ QX_e)  (Q_e = adjoint of hbar^t at j),
//   Xbt copied to the k slots; P_e = Fbt * Xbar_e  (routed to h_j), added to
//   the P_e already stored when accP is set.
// With rpos (the loss gradient in positions): rbar_e = sum_t Fbar . F'_e depends
// on r_e through B'(r_e) too, so rpos_e += rt_e Fbar . F''_e, F'' = B''(r_e) W_b.
template <int VPL, int KC>
__global__ void edge_p3_kernel(const float* __restrict__ B, const float* __restrict__ dB, int nb,
                               const float* __restrict__ Wb, const float* __restrict__ h, const int* __restrict__ ej,
                               const int* __restrict__ pos, long long Ne, int d, const float* __restrict__ Xbar,
                               const float* __restrict__ hht, const float* __restrict__ rt, float* __restrict__ Xbts,
                               float* __restrict__ P, const float* __restrict__ QX, int accP,
                               const float* __restrict__ d2B, float* __restrict__ rpos, float* __restrict__ Xrow) {
  extern __shared__ float sW[];
  load_lds(sW, Wb, nb * d);
  JANUS_WAVE_LOOP(e, Ne) {
    const float bl = basis_lane(B, e, nb, l), dbl = basis_lane(dB, e, nb, l);
    const long long j = ej[e];
    const float r = rt[e];
    float q[VPL], hj[VPL], xb[VPL], qx[VPL];
    if (hht) ld_row<VPL>(hht + j * d, l, q); else zero_row<VPL>(q);
    ld_row<VPL>(h + j * d, l, hj);
    ld_row<VPL>(Xbar + e * d, l, xb);
    if (QX) ld_row<VPL>(QX + e * d, l, qx); else zero_row<VPL>(qx);
    float F[VPL], Fp[VPL];
    filter_rows2<VPL>(bl, dbl, sW, nb, d, l, F, Fp);
    float X[VPL], p[VPL];
    if (accP) ld_row<VPL>(P + e * d, l, p); else zero_row<VPL>(p);
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const float fbt = r * Fp[v];
      X[v] = q[v] * F[v] + fbt * hj[v] + qx[v];
      p[v] += fbt * xb[v];
    }
    st_row<VPL>(P + e * d, l, p);
#pragma unroll
    for (int c = 0; c < KC; ++c) st_row<VPL>(Xbts + (long long)pos[e * KC + c] * d, l, X);
    if (Xrow) st_row<VPL>(Xrow + e * d, l, X);   // Xbt per edge (routing on the edge tokens)
    if (rpos) {
      float F2[VPL];
      filter_row<VPL>(basis_lane(d2B, e, nb, l), sW, nb, d, l, F2);
      float s2 = 0.f;
#pragma unroll
      for (int v = 0; v < VPL; ++v) s2 += xb[v] * hj[v] * F2[v];
      s2 = wave_sum(s2);
      if (l == 0) rpos[e] += r * s2;
    }
  }
}

// Phase 3 per atom: gate adjoints g3_ec = Ybt[pos] . hbar^{t+1}_i and
// hht^{t+1}_i = hht^t_i + sum_{e in seg(i)} sum_c g_ec Ybt[pos[e, c]].
template <int VPL, int KC>
__global__ void combine_p3_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos,
                                  const float* __restrict__ gate, const float* __restrict__ Ybt,
                                  const float* __restrict__ hbar_next, const float* __restrict__ hht, int N, int d,
                                  float* __restrict__ g3, float* __restrict__ hht_next) {
  JANUS_WAVE_LOOP(i, N) {
    float mb[VPL], acc[VPL];
    ld_row<VPL>(hbar_next + i * d, l, mb);
    if (hht) ld_row<VPL>(hht + i * d, l, acc); else zero_row<VPL>(acc);
    const long long f0 = (long long)rowptr[i] * KC, f1 = (long long)rowptr[i + 1] * KC;
    long long f = f0;
    // eight slot rows (of consecutive edges) in flight per step; each row's dot
    // product with hbar goes to lane u of the g3 store
    for (; f + 8 <= f1; f += 8) {
      float y[8][VPL], g[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        ld_row<VPL>(Ybt + (long long)pos[f + u] * d, l, y[u]);
        g[u] = gate[f + u];
      }
      float o = 0.f;
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        float su = 0.f;
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          su += y[u][v] * mb[v];
          acc[v] += g[u] * y[u][v];
        }
        su = wave_sum(su);
        o = l == u ? su : o;
      }
      if (l < 8) g3[f + l] = o;
    }
    for (; f < f1; ++f) {
      float y[VPL];
      ld_row<VPL>(Ybt + (long long)pos[f] * d, l, y);
      const float g = gate[f];
      float su = 0.f;
#pragma unroll
      for (int v = 0; v < VPL; ++v) {
        su += y[v] * mb[v];
        acc[v] += g * y[v];
      }
      su = wave_sum(su);
      if (l == 0) g3[f] = su;
    }
    st_row<VPL>(hht_next + i * d, l, acc);
  }
}

// Phase 4 per edge: Xt_e = sum_c Xt_slot (+ Xadd_e); Ft_e = Xt * h_j + Q_e * Xbar_e
// (Q_e from the double backward); P_e = Xt * F_e (routed to h_j).
// With rpos: F_e = B(r_e) W_b, so rpos_e += Ft . F'_e.
template <int VPL, int KC>
__global__ void edge_p4_kernel(const float* __restrict__ B, int nb, const float* __restrict__ Wb,
                               const float* __restrict__ h, const int* __restrict__ ej, const int* __restrict__ pos,
                               long long Ne, int d, const float* __restrict__ Xts, const float* __restrict__ Xbar,
                               const float* __restrict__ hht, float* __restrict__ Ft, float* __restrict__ P,
                               float* __restrict__ XT, const float* __restrict__ dB, float* __restrict__ rpos,
                               const float* __restrict__ Xadd) {
  extern __shared__ float sW[];
  load_lds(sW, Wb, nb * d);
  JANUS_WAVE_LOOP(e, Ne) {
    const float bl = basis_lane(B, e, nb, l);
    const long long j = ej[e];
    float xt[VPL], hj[VPL], q[VPL], xb[VPL];
    sum_slots<VPL, KC>(Xts, pos, e, d, l, xt);
    if (Xadd) {   // the router's part of Xt (routing on the edge tokens)
      float xa[VPL];
      ld_row<VPL>(Xadd + e * d, l, xa);
      add_row<VPL>(xt, xa);
    }
    ld_row<VPL>(h + j * d, l, hj);
    if (hht) ld_row<VPL>(hht + j * d, l, q); else zero_row<VPL>(q);
    ld_row<VPL>(Xbar + e * d, l, xb);
    float F[VPL];
    filter_row<VPL>(bl, sW, nb, d, l, F);
    float ft[VPL], p[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      ft[v] = xt[v] * hj[v] + q[v] * xb[v];
      p[v] = xt[v] * F[v];
    }
    st_row<VPL>(Ft + e * d, l, ft);
    st_row<VPL>(P + e * d, l, p);
    if (XT) st_row<VPL>(XT + e * d, l, xt);
    if (rpos) {
      float Fp[VPL];
      filter_row<VPL>(basis_lane(dB, e, nb, l), sW, nb, d, l, Fp);
      float s1 = 0.f;
#pragma unroll
      for (int v = 0; v < VPL; ++v) s1 += ft[v] * Fp[v];
      s1 = wave_sum(s1);
      if (l == 0) rpos[e] += s1;
    }
  }
}

}  // namespace janus
