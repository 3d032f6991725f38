// Edge- and atom-level kernels of the training step (wave64, one wave per
// edge or per atom; lane l owns feature columns l, l + 64, ...).
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
#pragma once

#include "common.h"

namespace janus {

template <int VPL>
__device__ __forceinline__ void filter_row(const float* __restrict__ Bv, const float* sW, int nb, int d, int l,
                                           float (&F)[VPL]) {
#pragma unroll
  for (int v = 0; v < VPL; ++v) F[v] = 0.f;
  for (int n = 0; n < nb; ++n) {
    const float b = Bv[n];
#pragma unroll
    for (int v = 0; v < VPL; ++v) F[v] += b * sW[n * d + v * 64 + l];
  }
}

__device__ __forceinline__ void load_lds(float* s, const float* g, int n) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) s[i] = g[i];
  __syncthreads();
}

#define JANUS_WAVE_LOOP(var, count)                                                     \
  const int l = threadIdx.x & 63;                                                       \
  const long long nw_ = (long long)gridDim.x * (blockDim.x >> 6);                       \
  for (long long var = (long long)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); \
       var < (count); var += nw_)

// Phase 1: X_e = F_e * h_j (+ Q_e, the triplet messages of e when present),
// written to the slots of its k experts.
template <int VPL>
__global__ void dispatch_x_kernel(const float* __restrict__ B, int nb, const float* __restrict__ Wb,
                                  const float* __restrict__ h, const int* __restrict__ ej,
                                  const int* __restrict__ pos, int k, long long Ne, int d, float* __restrict__ Xs,
                                  const float* __restrict__ Q) {
  extern __shared__ float sW[];
  load_lds(sW, Wb, nb * d);
  JANUS_WAVE_LOOP(e, Ne) {
    float F[VPL];
    filter_row<VPL>(B + e * nb, sW, nb, d, l, F);
    const float* hj = h + (long long)ej[e] * d;
    float X[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) X[v] = F[v] * hj[v * 64 + l] + (Q ? Q[e * d + v * 64 + l] : 0.f);
    for (int c = 0; c < k; ++c) {
      float* o = Xs + (long long)pos[e * k + c] * d;
#pragma unroll
      for (int v = 0; v < VPL; ++v) o[v * 64 + l] = X[v];
    }
  }
}

// Phase 1: h'_i = h_i + sum_{e in seg(i)} sum_c Yg[pos[e, c]]  (Yg already gated).
template <int VPL>
__global__ void combine_fwd_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos, int k,
                                   const float* __restrict__ Yg, const float* __restrict__ h, int N, int d,
                                   float* __restrict__ hn) {
  JANUS_WAVE_LOOP(i, N) {
    float acc[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) acc[v] = h[i * d + v * 64 + l];
    const int e0 = rowptr[i], e1 = rowptr[i + 1];
    for (int e = e0; e < e1; ++e)
      for (int c = 0; c < k; ++c) {
        const float* y = Yg + (long long)pos[(long long)e * k + c] * d;
#pragma unroll
        for (int v = 0; v < VPL; ++v) acc[v] += y[v * 64 + l];
      }
#pragma unroll
    for (int v = 0; v < VPL; ++v) hn[i * d + v * 64 + l] = acc[v];
  }
}

// Slot rows of the adjoint arriving at the messages: out[pos[e, c]] = (g_ec) * src[i(e)].
template <int VPL>
__global__ void gather_atom_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos, int k,
                                   const float* __restrict__ gate, const float* __restrict__ src, int N, int d,
                                   float* __restrict__ out) {
  JANUS_WAVE_LOOP(i, N) {
    float s[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) s[v] = src[i * d + v * 64 + l];
    const int e0 = rowptr[i], e1 = rowptr[i + 1];
    for (int e = e0; e < e1; ++e)
      for (int c = 0; c < k; ++c) {
        const long long f = (long long)e * k + c;
        const float g = gate ? gate[f] : 1.f;
        float* o = out + (long long)pos[f] * d;
#pragma unroll
        for (int v = 0; v < VPL; ++v) o[v * 64 + l] = g * s[v];
      }
  }
}

// Phase 2 per edge: Xbar_e = sum_c Xbar_slot; Fbar = Xbar * h_j;
// rbar_e += Fbar . F'_e; P_e = Xbar * F_e (routed to h_j by scatter_rev).
template <int VPL>
__global__ void edge_p2_kernel(const float* __restrict__ B, const float* __restrict__ dB, int nb,
                               const float* __restrict__ Wb, const float* __restrict__ h, const int* __restrict__ ej,
                               const int* __restrict__ pos, int k, long long Ne, int d,
                               const float* __restrict__ Xbs, float* __restrict__ Xbar, float* __restrict__ Fbar,
                               float* __restrict__ rbar, float* __restrict__ P) {
  extern __shared__ float sW[];
  load_lds(sW, Wb, nb * d);
  JANUS_WAVE_LOOP(e, Ne) {
    float xb[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) xb[v] = 0.f;
    for (int c = 0; c < k; ++c) {
      const float* y = Xbs + (long long)pos[e * k + c] * d;
#pragma unroll
      for (int v = 0; v < VPL; ++v) xb[v] += y[v * 64 + l];
    }
    float F[VPL], Fp[VPL];
    filter_row<VPL>(B + e * nb, sW, nb, d, l, F);
    filter_row<VPL>(dB + e * nb, sW, nb, d, l, Fp);
    const float* hj = h + (long long)ej[e] * d;
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const long long o = e * d + v * 64 + l;
      const float fb = xb[v] * hj[v * 64 + l];
      Xbar[o] = xb[v];
      Fbar[o] = fb;
      P[o] = xb[v] * F[v];
      s += fb * Fp[v];
    }
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
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      acc[v] = base0 ? base0[a * d + v * 64 + l] : 0.f;
      if (base1) acc[v] += base1[a * d + v * 64 + l];
    }
    const int e0 = rowptr[a], e1 = rowptr[a + 1];
    for (int e = e0; e < e1; ++e) {
      const float* p = P + (long long)rev[e] * d;
#pragma unroll
      for (int v = 0; v < VPL; ++v) acc[v] += p[v * 64 + l];
    }
#pragma unroll
    for (int v = 0; v < VPL; ++v) out[a * d + v * 64 + l] = acc[v];
  }
}

// Phase 3 per edge (adjoints of the force backward):
//   Fbt = rt_e F'_e,  Xbt = Q_e * F_e + Fbt * h_j  (Q_e = adjoint of hbar^t at j),
//   Xbt copied to the k slots; P_e = Fbt * Xbar_e  (routed to h_j).
template <int VPL>
__global__ void edge_p3_kernel(const float* __restrict__ B, const float* __restrict__ dB, int nb,
                               const float* __restrict__ Wb, const float* __restrict__ h, const int* __restrict__ ej,
                               const int* __restrict__ pos, int k, long long Ne, int d, const float* __restrict__ Xbar,
                               const float* __restrict__ hht, const float* __restrict__ rt, float* __restrict__ Xbts,
                               float* __restrict__ P, const float* __restrict__ QX) {
  extern __shared__ float sW[];
  load_lds(sW, Wb, nb * d);
  JANUS_WAVE_LOOP(e, Ne) {
    float F[VPL], Fp[VPL];
    filter_row<VPL>(B + e * nb, sW, nb, d, l, F);
    filter_row<VPL>(dB + e * nb, sW, nb, d, l, Fp);
    const long long j = ej[e];
    const float r = rt[e];
    float X[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const int col = v * 64 + l;
      const float fbt = r * Fp[v];
      const float q = hht ? hht[j * d + col] : 0.f;
      X[v] = q * F[v] + fbt * h[j * d + col] + (QX ? QX[e * d + col] : 0.f);
      P[e * d + col] = fbt * Xbar[e * d + col];
    }
    for (int c = 0; c < k; ++c) {
      float* o = Xbts + (long long)pos[e * k + c] * d;
#pragma unroll
      for (int v = 0; v < VPL; ++v) o[v * 64 + l] = X[v];
    }
  }
}

// Phase 3 per atom: gate adjoints g3_ec = Ybt[pos] . hbar^{t+1}_i and
// hht^{t+1}_i = hht^t_i + sum_{e in seg(i)} sum_c g_ec Ybt[pos[e, c]].
template <int VPL>
__global__ void combine_p3_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos, int k,
                                  const float* __restrict__ gate, const float* __restrict__ Ybt,
                                  const float* __restrict__ hbar_next, const float* __restrict__ hht, int N, int d,
                                  float* __restrict__ g3, float* __restrict__ hht_next) {
  JANUS_WAVE_LOOP(i, N) {
    float mb[VPL], acc[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      mb[v] = hbar_next[i * d + v * 64 + l];
      acc[v] = hht ? hht[i * d + v * 64 + l] : 0.f;
    }
    const int e0 = rowptr[i], e1 = rowptr[i + 1];
    for (int e = e0; e < e1; ++e)
      for (int c = 0; c < k; ++c) {
        const long long f = (long long)e * k + c;
        const float* y = Ybt + (long long)pos[f] * d;
        const float g = gate[f];
        float s = 0.f;
#pragma unroll
        for (int v = 0; v < VPL; ++v) {
          const float yv = y[v * 64 + l];
          s += yv * mb[v];
          acc[v] += g * yv;
        }
        s = wave_sum(s);
        if (l == 0) g3[f] = s;
      }
#pragma unroll
    for (int v = 0; v < VPL; ++v) hht_next[i * d + v * 64 + l] = acc[v];
  }
}

// Phase 4 per edge: Xt_e = sum_c Xt_slot; Ft_e = Xt * h_j + Q_e * Xbar_e
// (Q_e from the double backward); P_e = Xt * F_e (routed to h_j).
template <int VPL>
__global__ void edge_p4_kernel(const float* __restrict__ B, int nb, const float* __restrict__ Wb,
                               const float* __restrict__ h, const int* __restrict__ ej, const int* __restrict__ pos,
                               int k, long long Ne, int d, const float* __restrict__ Xts,
                               const float* __restrict__ Xbar, const float* __restrict__ hht,
                               float* __restrict__ Ft, float* __restrict__ P, float* __restrict__ XT) {
  extern __shared__ float sW[];
  load_lds(sW, Wb, nb * d);
  JANUS_WAVE_LOOP(e, Ne) {
    float xt[VPL];
#pragma unroll
    for (int v = 0; v < VPL; ++v) xt[v] = 0.f;
    for (int c = 0; c < k; ++c) {
      const float* y = Xts + (long long)pos[e * k + c] * d;
#pragma unroll
      for (int v = 0; v < VPL; ++v) xt[v] += y[v * 64 + l];
    }
    float F[VPL];
    filter_row<VPL>(B + e * nb, sW, nb, d, l, F);
    const long long j = ej[e];
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const int col = v * 64 + l;
      const float q = hht ? hht[j * d + col] : 0.f;
      Ft[e * d + col] = xt[v] * h[j * d + col] + q * Xbar[e * d + col];
      P[e * d + col] = xt[v] * F[v];
      if (XT) XT[e * d + col] = xt[v];
    }
  }
}

}  // namespace janus
