// Routing on the evolving edge tokens (paper Sec. "Sparse mixture-of-experts
// (MoE) routing", with the router a linear layer on the token): per block t
//   l_e = (Pc[Z_i] + Pn[Z_j]) + X_e Wr + beta,   top-k of the fp32 logits,
//   gates g_ec = p_e[x_c] with p_e = softmax(l_e) over all E experts,
// so the gates move with X_e and the four phases carry their derivatives (mbar_i,
// mt_i and the tangent below are the atom's; with self-attention they are the edge's
// own message adjoints and tangent, read through identity index maps):
//   phase 2 (forces):  gbar_c = <mbar_i, Y_c>,  lbar = J(p)^T gbar,
//                      Xbar_e += Wr lbar   (J(p) = diag(p) - p p^T);
//   phase 3 (double backward), from Xh = the loss adjoint of Xbar:
//                      lh = Xh Wr,  gh_c = (J(p) lh)_{x_c}  (-> hht_i += gh_c Y_c,
//                      and the primal Y_c gains gh_c mbar_i in phase 4),
//                      P3_z = lh_z (gbar~_z - s) - gbar~_z <lh, p>,  s = sum_c g_c gbar_c
//                      (the loss adjoint of p through lbar), dWr += Xh^T lbar;
//   phase 4 (final backward):  lt = J(p)^T (g3~ + g4~ + P3), g4_c = <mt_i, Y_c>,
//                      Xt_e += Wr lt,  dWr += X^T lt,  Pc/Pn from lt.
// (gbar~ is gbar scattered to the chosen experts.)  Y_c is the expert output
// before gating; logit rows are padded to Ep (a multiple of 16) columns.
#pragma once

#include "edge.h"

namespace janus {

// WrP [d, Ep]: Wr [d, E] with zero columns E..Ep-1.
__global__ void wr_pad_kernel(const float* __restrict__ Wr, int d, int E, int Ep, float* __restrict__ WrP) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (long long)d * Ep) return;
  const int r = (int)(q / Ep), c = (int)(q - (long long)r * Ep);
  WrP[q] = c < E ? Wr[(long long)r * E + c] : 0.f;
}

// G [d, E] += GP [d, Ep] (first E columns).
__global__ void wr_unpad_add_kernel(const float* __restrict__ GP, int d, int E, int Ep, float* __restrict__ G) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (long long)d * E) return;
  const int r = (int)(q / E), c = (int)(q - (long long)r * E);
  G[q] += GP[(long long)r * Ep + c];
}

// Per edge: logits l_x = (Pc[Z_i, x] + Pn[Z_j, x]) + XW[e, x] + beta_x (fp32), the top
// k in descending order (lower index first on ties), the full softmax p (float64,
// stored fp32), the chosen gates, and the margin l_(k) - l_(k+1) of the decision.
__global__ void feat_route_kernel(const float* __restrict__ XW, const int* __restrict__ species,
                                  const int* __restrict__ ei, const int* __restrict__ ej,
                                  const float* __restrict__ Pc, const float* __restrict__ Pn,
                                  const float* __restrict__ beta, long long Ne, int E, int Ep, int k,
                                  int* __restrict__ eid, float* __restrict__ gate, float* __restrict__ prob,
                                  float* __restrict__ gap) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const float* pc = Pc + (long long)species[ei[e]] * E;
  const float* pn = Pn + (long long)species[ej[e]] * E;
  const float* xw = XW + e * Ep;
  auto logit = [&](int x) { return (pc[x] + pn[x]) + xw[x] + beta[x]; };
  // k passes of an arg-max that skips the experts already taken
  int chosen[kMaxTopK];
  float lk = 0.f;
  for (int c = 0; c < k; ++c) {
    int best = -1;
    float bv = 0.f;
    for (int x = 0; x < E; ++x) {
      bool taken = false;
      for (int q = 0; q < c; ++q) taken |= chosen[q] == x;
      if (taken) continue;
      const float v = logit(x);
      if (best < 0 || v > bv) {
        best = x;
        bv = v;
      }
    }
    chosen[c] = best;
    lk = bv;
  }
  float next = -INFINITY;
  for (int x = 0; x < E; ++x) {
    bool taken = false;
    for (int q = 0; q < k; ++q) taken |= chosen[q] == x;
    if (!taken) next = fmaxf(next, logit(x));
  }
  double mx = -INFINITY;
  for (int x = 0; x < E; ++x) mx = fmax(mx, (double)logit(x));
  double z = 0.0;
  for (int x = 0; x < E; ++x) z += exp((double)logit(x) - mx);
  for (int x = 0; x < Ep; ++x) prob[e * Ep + x] = x < E ? (float)(exp((double)logit(x) - mx) / z) : 0.f;
  for (int c = 0; c < k; ++c) {
    eid[e * k + c] = chosen[c];
    gate[e * k + c] = (float)(exp((double)logit(chosen[c]) - mx) / z);
  }
  if (gap) gap[e] = k < E ? lk - next : INFINITY;
}

// h'_i = h_i + sum_{e in seg(i)} sum_c g_ec Y[pos[e, c]]  (Y before gating; h may be
// null: zero).  With the identity segments (rowptr[e] = e) it forms the gated
// message of every edge, the attention layer's tokens.
template <int VPL, int KC>
__global__ void combine_fwd_gated_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos,
                                         const float* __restrict__ gate, const float* __restrict__ Y,
                                         const float* __restrict__ h, long long N, int d, float* __restrict__ hn) {
  JANUS_WAVE_LOOP(i, N) {
    float acc[VPL];
    if (h) ld_row<VPL>(h + i * d, l, acc); else zero_row<VPL>(acc);
    const long long f1 = (long long)rowptr[i + 1] * KC;
    long long f = (long long)rowptr[i] * KC;
    for (; f + 4 <= f1; f += 4) {
      float y[4][VPL], g[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        ld_row<VPL>(Y + (long long)pos[f + u] * d, l, y[u]);
        g[u] = gate[f + u];
      }
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int v = 0; v < VPL; ++v) acc[v] += g[u] * y[u][v];
    }
    for (; f < f1; ++f) {
      float y[VPL];
      ld_row<VPL>(Y + (long long)pos[f] * d, l, y);
      const float g = gate[f];
#pragma unroll
      for (int v = 0; v < VPL; ++v) acc[v] += g * y[v];
    }
    st_row<VPL>(hn + i * d, l, acc);
  }
}

// <a, Y[pos[e, c]]> for the k slots of edge e (wave-uniform results).
template <int VPL, int KC>
__device__ __forceinline__ void slot_dots(const float* __restrict__ Y, const int* __restrict__ pos, long long e,
                                          int d, int l, const float (&a)[VPL], float (&out)[KC]) {
  float y[KC][VPL];
#pragma unroll
  for (int c = 0; c < KC; ++c) ld_row<VPL>(Y + (long long)pos[e * KC + c] * d, l, y[c]);
#pragma unroll
  for (int c = 0; c < KC; ++c) {
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < VPL; ++v) s += a[v] * y[c][v];
    out[c] = wave_sum(s);
  }
}

// Phase 2 per edge: gbar_c = <mbar_i, Y_c> (kept), lbar = J(p)^T gbar [Ep].
template <int VPL, int KC>
__global__ void feat_p2_kernel(const int* __restrict__ ei, const int* __restrict__ pos, const int* __restrict__ eid,
                               const float* __restrict__ gate, const float* __restrict__ prob, int E, int Ep,
                               const float* __restrict__ mbar, const float* __restrict__ Y, long long Ne, int d,
                               float* __restrict__ gbar, float* __restrict__ lbar) {
  JANUS_WAVE_LOOP(e, Ne) {
    float m[VPL], gb[KC];
    ld_row<VPL>(mbar + (long long)ei[e] * d, l, m);
    slot_dots<VPL, KC>(Y, pos, e, d, l, m, gb);
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < KC; ++c) s += gate[e * KC + c] * gb[c];
    if (l < KC) {
      float v = 0.f;
#pragma unroll
      for (int c = 0; c < KC; ++c) v = l == c ? gb[c] : v;
      gbar[e * KC + l] = v;
    }
    if (l < Ep) {
      float gt = 0.f;   // gbar scattered to the chosen experts
#pragma unroll
      for (int c = 0; c < KC; ++c) gt = eid[e * KC + c] == l ? gb[c] : gt;
      lbar[e * Ep + l] = l < E ? prob[e * Ep + l] * (gt - s) : 0.f;
    }
  }
}

// Phase 3 per edge (one thread): from lh = Xh Wr [Ep],
//   gh_c = g_c (lh_{x_c} - <p, lh>),  P3_z = lh_z (gbar~_z - s) - gbar~_z <p, lh>.
__global__ void feat_p3_kernel(const int* __restrict__ eid, const float* __restrict__ gate,
                               const float* __restrict__ prob, const float* __restrict__ gbar,
                               const float* __restrict__ lh, long long Ne, int E, int Ep, int k,
                               float* __restrict__ gh, float* __restrict__ P3) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const float* p = prob + e * Ep;
  const float* L = lh + e * Ep;
  double mu = 0.0;
  for (int x = 0; x < E; ++x) mu += (double)p[x] * L[x];
  double s = 0.0;
  for (int c = 0; c < k; ++c) s += (double)gate[e * k + c] * gbar[e * k + c];
  for (int c = 0; c < k; ++c) {
    const int x = eid[e * k + c];
    gh[e * k + c] = (float)((double)gate[e * k + c] * ((double)L[x] - mu));
  }
  for (int z = 0; z < Ep; ++z) {
    double gz = 0.0;
    for (int c = 0; c < k; ++c) gz = eid[e * k + c] == z ? (double)gbar[e * k + c] : gz;
    P3[e * Ep + z] = z < E ? (float)((double)L[z] * (gz - s) - gz * mu) : 0.f;
  }
}

// Phase 3 per atom: hht'_i += sum_{e in seg(i)} sum_c gh_ec Y[pos[e, c]] (with the
// identity segments, per edge: the gates' part of the message tangent).
template <int VPL, int KC>
__global__ void feat_hht_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos,
                                const float* __restrict__ gh, const float* __restrict__ Y, long long N, int d,
                                float* __restrict__ hht) {
  JANUS_WAVE_LOOP(i, N) {
    float acc[VPL];
    ld_row<VPL>(hht + i * d, l, acc);
    const long long f1 = (long long)rowptr[i + 1] * KC;
    for (long long f = (long long)rowptr[i] * KC; f < f1; ++f) {
      float y[VPL];
      ld_row<VPL>(Y + (long long)pos[f] * d, l, y);
      const float g = gh[f];
#pragma unroll
      for (int v = 0; v < VPL; ++v) acc[v] += g * y[v];
    }
    st_row<VPL>(hht + i * d, l, acc);
  }
}

// Phase 4: slot rows of the loss adjoint of the expert outputs,
//   out[pos[e, c]] = g_ec mt_i + gh_ec mbar_i
// (with the identity segments and per-edge mt, mbar: the attention layer's message
// adjoints).
template <int VPL, int KC>
__global__ void gather_feat_kernel(const int* __restrict__ rowptr, const int* __restrict__ pos,
                                   const float* __restrict__ gate, const float* __restrict__ mt,
                                   const float* __restrict__ gh, const float* __restrict__ mbar, long long N,
                                   int d, float* __restrict__ out) {
  JANUS_WAVE_LOOP(i, N) {
    float a[VPL], b[VPL];
    ld_row<VPL>(mt + i * d, l, a);
    ld_row<VPL>(mbar + i * d, l, b);
    const long long f1 = (long long)rowptr[i + 1] * KC;
    for (long long f = (long long)rowptr[i] * KC; f < f1; ++f) {
      const float g = gate[f], q = gh[f];
      float o[VPL];
#pragma unroll
      for (int v = 0; v < VPL; ++v) o[v] = g * a[v] + q * b[v];
      st_row<VPL>(out + (long long)pos[f] * d, l, o);
    }
  }
}

// Phase 4 per edge: g4_c = <mt_i, Y_c>; pt = (g3 + g4)~ + P3; lt = J(p)^T pt
// into lt [Ep] (padded) and lte [E] (the router tables' per-edge adjoint).
template <int VPL, int KC>
__global__ void feat_p4_kernel(const int* __restrict__ ei, const int* __restrict__ pos, const int* __restrict__ eid,
                               const float* __restrict__ prob, int E, int Ep, const float* __restrict__ mt,
                               const float* __restrict__ Y, const float* __restrict__ g3,
                               const float* __restrict__ P3, long long Ne, int d, float* __restrict__ lt,
                               float* __restrict__ lte) {
  JANUS_WAVE_LOOP(e, Ne) {
    float m[VPL], g4[KC];
    ld_row<VPL>(mt + (long long)ei[e] * d, l, m);
    slot_dots<VPL, KC>(Y, pos, e, d, l, m, g4);
    float pt = 0.f, pz = 0.f;
    if (l < E) {
      pz = prob[e * Ep + l];
      pt = P3[e * Ep + l];
#pragma unroll
      for (int c = 0; c < KC; ++c)
        if (eid[e * KC + c] == l) pt += g3[e * KC + c] + g4[c];
    }
    const float mu = wave_sum(pz * pt);
    const float v = l < E ? pz * (pt - mu) : 0.f;
    if (l < Ep) lt[e * Ep + l] = v;
    if (l < E) lte[e * E + l] = v;
  }
}

}  // namespace janus
