#pragma once
// Kernels, epilogues, weight layout and workspace plan of the training step
// (included once, by driver.hip).  The step runs the four phases of the
// double-backward schedule (paper Sec. "Runtime for multi-phase
// double-backward execution"): forward to the energy, first backward to the
// forces, double backward of the force loss, final backward of the energy
// loss.  Gradient contributions of the double and final backward passes to
// the same weight are accumulated in a fixed order.
#include <cstdio>
#include <cstring>
#include <string>
#include <vector>

#include "edge.h"
#include "internal.h"
#include "kernels.h"
#include "route.h"
#include "tri.h"
#include "attn.h"
#include "attn_tiled.h"
#include "feat_route.h"

namespace janus {

// ------------------------------------------------------------ small kernels

// Bit 1: bad species / offsets; bit 2: bad CSR; bit 4: bad edge indices or reverse map.
__global__ void validate_atoms_kernel(const int* __restrict__ species, int N, int nsp, const int* __restrict__ rowptr,
                                      const int* __restrict__ ei, long long Ne, const int* __restrict__ offsets, int S,
                                      int* __restrict__ flag) {
  const int a = blockIdx.x * blockDim.x + threadIdx.x;
  if (a < S && offsets[a] >= offsets[a + 1]) atomicOr(flag, 1);   // every structure holds an atom
  if (a > N) return;
  int bad = 0;
  if (a == 0 && rowptr[0] != 0) bad |= 2;
  if (a == N) {
    if (rowptr[N] != Ne) bad |= 2;
  } else {
    if (species[a] < 0 || species[a] >= nsp) bad |= 1;
    const int e0 = rowptr[a], e1 = rowptr[a + 1];
    if (e0 < 0 || e1 < e0 || e1 > Ne) {
      bad |= 2;
    } else {
      for (int e = e0; e < e1; ++e)
        if (ei[e] != a) { bad |= 2; break; }
    }
  }
  if (bad) atomicOr(flag, bad);
}

__global__ void validate_edges_kernel(const int* __restrict__ ei, const int* __restrict__ ej,
                                      const int8_t* __restrict__ shift, const int* __restrict__ rev,
                                      const int* __restrict__ sid, int N, long long Ne, int* __restrict__ flag) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const int i = ei[e], j = ej[e], r = rev[e];
  bool ok = i >= 0 && i < N && j >= 0 && j < N && r >= 0 && r < Ne;
  if (ok) {
    ok = rev[r] == e && ei[r] == j && ej[r] == i && sid[i] == sid[j] && shift[3 * r] == -shift[3 * e] &&
         shift[3 * r + 1] == -shift[3 * e + 1] && shift[3 * r + 2] == -shift[3 * e + 2] &&
         !(i == j && shift[3 * e] == 0 && shift[3 * e + 1] == 0 && shift[3 * e + 2] == 0);
  }
  if (!ok) atomicOr(flag, 4);
}

// Per-atom readout energy eps_i = w_o2 . SiLU(z_i)  (z = h^T W_o1).
template <int VPL>
__global__ void readout_kernel(const float* __restrict__ z, const float* __restrict__ wo2, int N, int d,
                               float* __restrict__ eps) {
  JANUS_WAVE_LOOP(i, N) {
    float s = 0.f;
#pragma unroll
    for (int v = 0; v < VPL; ++v) s += silu(z[i * d + v * 64 + l]) * wo2[v * 64 + l];
    s = wave_sum(s);
    if (l == 0) eps[i] = s;
  }
}

// E_s = sum of eps over the atoms of s, accumulated in float64.
__global__ void energy_kernel(const float* __restrict__ eps, const int* __restrict__ offsets, int S,
                              double* __restrict__ Ed, float* __restrict__ E) {
  JANUS_WAVE_LOOP(s, S) {
    double acc = 0.0;
    for (int a = offsets[s] + l; a < offsets[s + 1]; a += 64) acc += (double)eps[a];
    acc = wave_sum_d(acc);
    if (l == 0) {
      Ed[s] = acc;
      E[s] = (float)acc;
    }
  }
}

// F_a = sum_{e in seg(a)} (G_e - G_rev(e)),  G_e = rbar_e u_e = dE/dd_e.
// With the three-body term, G_e gains the triplet displacement adjoint gvec[e].
__global__ void force_kernel(const int* __restrict__ rowptr, const int* __restrict__ rev,
                             const float* __restrict__ rbar, const float4* __restrict__ geo,
                             const float4* __restrict__ gvec, int N, float* __restrict__ F) {
  // one wave per atom: lane l sums the edges l, l + 64, ... of the atom in
  // order, then the lanes are added in a fixed butterfly (float64 throughout)
  JANUS_WAVE_LOOP(a, N) {
    double fx = 0, fy = 0, fz = 0;
    const int e1 = rowptr[a + 1];
    for (int e = rowptr[a] + l; e < e1; e += kWave) {
      const int er = rev[e];
      const float4 u = geo[e], ur = geo[er];
      const double g = rbar[e], gr = rbar[er];
      fx += g * u.x - gr * ur.x;
      fy += g * u.y - gr * ur.y;
      fz += g * u.z - gr * ur.z;
      if (gvec) {
        const float4 v = gvec[e], vr = gvec[er];
        fx += (double)v.x - vr.x;
        fy += (double)v.y - vr.y;
        fz += (double)v.z - vr.z;
      }
    }
    fx = wave_sum_d(fx);
    fy = wave_sum_d(fy);
    fz = wave_sum_d(fz);
    if (l == 0) {
      F[3 * a] = (float)fx;
      F[3 * a + 1] = (float)fy;
      F[3 * a + 2] = (float)fz;
    }
  }
}

// Loss gradient in the positions (paper Sec. "MatRIS": forces and stresses are
// derivatives of E, so the loss depends on R through E, F = -dE/dR and sigma).
// Per edge, with G_e = rbar_e u_e = dE/dd_e:
//   L sees G_e through F_i (+G_e), F_j (-G_e) and sigma_s (G_e d_e^T / V_s), so
//   its adjoint is gt_e = phi_i - phi_j + Psi_s d_e;
//   u_e = d_e / r_e carries rbar_e gt_e, sigma's own d_e carries Psi_s^T G_e;
//   rpos_e (accumulated by the double and final backward) is dL/dr_e through
//   the basis B(r_e) and its derivative B'(r_e):
//   dL/dd_e = rpos_e u_e + rbar_e (gt_e - (gt_e . u_e) u_e) / r_e + rbar_e Psi_s^T u_e
//             (+ tpos_e, the bond-angle part, when the model has it),
// and dL/dR_a = sum over the edges e of a of (dL/dd_rev(e) - dL/dd_e) (d_e = R_j - R_i + n.L),
// one wave per atom, lanes over edges in order, a fixed butterfly, float64.
__device__ __forceinline__ void pos_edge_adjoint(int e, const int* __restrict__ ei, const int* __restrict__ ej,
                                                 const float* __restrict__ rbar, const float* __restrict__ rpos,
                                                 const float4* __restrict__ geo, const float* __restrict__ phi,
                                                 const float* __restrict__ Psi, const int* __restrict__ sid,
                                                 const float4* __restrict__ tpos, double (&a)[3]) {
  const int i = ei[e], j = ej[e];
  const float4 g = geo[e];
  const double u[3] = {g.x, g.y, g.z}, r = g.w;
  double gt[3];
  for (int k = 0; k < 3; ++k) gt[k] = (double)phi[3 * i + k] - (double)phi[3 * j + k];
  const float* P = Psi ? Psi + 9 * sid[i] : nullptr;
  if (P) {
    for (int k = 0; k < 3; ++k) gt[k] += r * ((double)P[3 * k] * u[0] + (double)P[3 * k + 1] * u[1] +
                                              (double)P[3 * k + 2] * u[2]);
  }
  const double rb = rbar[e], rp = rpos[e];
  const double gu = gt[0] * u[0] + gt[1] * u[1] + gt[2] * u[2];
  for (int k = 0; k < 3; ++k) a[k] = rp * u[k] + rb * (gt[k] - gu * u[k]) / r;
  if (P) {
    for (int k = 0; k < 3; ++k)
      a[k] += rb * ((double)P[k] * u[0] + (double)P[3 + k] * u[1] + (double)P[6 + k] * u[2]);
  }
  if (tpos) {   // the bond-angle part, per edge
    const float4 w = tpos[e];
    a[0] += w.x;
    a[1] += w.y;
    a[2] += w.z;
  }
}

__global__ void pos_grad_kernel(const int* __restrict__ rowptr, const int* __restrict__ rev,
                                const int* __restrict__ ei, const int* __restrict__ ej,
                                const float* __restrict__ rbar, const float* __restrict__ rpos,
                                const float4* __restrict__ geo, const float* __restrict__ phi,
                                const float* __restrict__ Psi, const int* __restrict__ sid,
                                const float4* __restrict__ tpos, int N, float* __restrict__ out) {
  JANUS_WAVE_LOOP(a, N) {
    double sx = 0, sy = 0, sz = 0;
    const int e1 = rowptr[a + 1];
    for (int e = rowptr[a] + l; e < e1; e += kWave) {
      double x[3], y[3];
      pos_edge_adjoint(e, ei, ej, rbar, rpos, geo, phi, Psi, sid, tpos, x);
      pos_edge_adjoint(rev[e], ei, ej, rbar, rpos, geo, phi, Psi, sid, tpos, y);
      sx += y[0] - x[0];
      sy += y[1] - x[1];
      sz += y[2] - x[2];
    }
    sx = wave_sum_d(sx);
    sy = wave_sum_d(sy);
    sz = wave_sum_d(sz);
    if (l == 0) {
      out[3 * a] = (float)sx;
      out[3 * a + 1] = (float)sy;
      out[3 * a + 2] = (float)sz;
    }
  }
}

// |det| of the lattice rows of one structure (its volume).
__device__ __forceinline__ double cell_volume(const float* __restrict__ c) {
  const double a0 = c[0], a1 = c[1], a2 = c[2], b0 = c[3], b1 = c[4], b2 = c[5], c0 = c[6], c1 = c[7], c2 = c[8];
  return fabs(a0 * (b1 * c2 - b2 * c1) - a1 * (b0 * c2 - b2 * c0) + a2 * (b0 * c1 - b1 * c0));
}

// Stress of every structure (one wave each), from G_e = dE/dd_e:
//   sigma_s[a][b] = (1/V_s) sum over the structure's edges of G_e,a d_e,b
// (a strain (I + eps) maps d_e to (I + eps) d_e).  The edges of a structure are
// contiguous: [rowptr[offsets[s]], rowptr[offsets[s+1]]).  fp64 accumulation in
// a fixed lane order.
__global__ void stress_kernel(const int* __restrict__ rowptr, const int* __restrict__ offsets,
                              const float* __restrict__ cell, const float* __restrict__ rbar,
                              const float4* __restrict__ geo, const float4* __restrict__ gvec, int S,
                              float* __restrict__ sig, float* __restrict__ out) {
  JANUS_WAVE_LOOP(s, S) {
    double w[9];
#pragma unroll
    for (int q = 0; q < 9; ++q) w[q] = 0.0;
    const int e1 = rowptr[offsets[s + 1]];
    for (int e = rowptr[offsets[s]] + l; e < e1; e += 64) {
      const float4 u = geo[e];
      double g[3] = {(double)rbar[e] * u.x, (double)rbar[e] * u.y, (double)rbar[e] * u.z};
      if (gvec) {
        const float4 v = gvec[e];
        g[0] += v.x;
        g[1] += v.y;
        g[2] += v.z;
      }
      const double dv[3] = {(double)u.x * u.w, (double)u.y * u.w, (double)u.z * u.w};
#pragma unroll
      for (int a = 0; a < 3; ++a)
#pragma unroll
        for (int b = 0; b < 3; ++b) w[3 * a + b] += g[a] * dv[b];
    }
    const double iv = 1.0 / cell_volume(cell + 9 * s);
#pragma unroll
    for (int q = 0; q < 9; ++q) w[q] = wave_sum_d(w[q]);
    if (l < 9) {
      double v = 0.0;
#pragma unroll
      for (int q = 0; q < 9; ++q) v = q == l ? w[q] : v;
      sig[9 * s + l] = (float)(v * iv);
      if (out) out[9 * s + l] = (float)(v * iv);
    }
  }
}

// Loss and adjoint seeds (one workgroup of 1024, fixed reduction order):
//   loss = w_E/S sum_s (E_s/n_s - Eref_s)^2 + w_F/(3N) sum_a |F_a - Fref_a|^2
//          [+ w_S/(9S) sum_s |sigma_s - Sref_s|^2]
//   lam_s = dloss/dE_s,  phi_a = dloss/dF_a,  Psi_s = (dloss/dsigma_s) / V_s.
// S, N: structures and atoms of this chunk; S_tot, N_tot: of the whole batch
// (the normalisation).  Writes this chunk's share of the loss to *loss_part.
// The stress term is skipped when Sref is null.
__global__ void loss_kernel(const double* __restrict__ Ed, const float* __restrict__ Eref,
                            const int* __restrict__ offsets, int S, const float* __restrict__ F,
                            const float* __restrict__ Fref, int N, int S_tot, int N_tot, float wE, float wF,
                            const float* __restrict__ sig, const float* __restrict__ Sref, float wS,
                            const float* __restrict__ cell, double* __restrict__ loss_part,
                            float* __restrict__ lam, float* __restrict__ phi, float* __restrict__ Psi) {
  __shared__ double red[1024];
  const int t = threadIdx.x;
  double se = 0.0, sf = 0.0, ss = 0.0;
  for (int s = t; s < S; s += 1024) {
    const double n = (double)(offsets[s + 1] - offsets[s]);
    const double de = Ed[s] / n - (double)Eref[s];
    se += de * de;
    lam[s] = (float)(2.0 * wE * de / ((double)S_tot * n));
    if (Sref) {
      const double iv = 1.0 / cell_volume(cell + 9 * s);
      for (int q = 0; q < 9; ++q) {
        const double ds = (double)sig[9 * s + q] - (double)Sref[9 * s + q];
        ss += ds * ds;
        Psi[9 * s + q] = (float)(2.0 * wS * ds / (9.0 * S_tot) * iv);
      }
    }
  }
  for (int q = t; q < 3 * N; q += 1024) {
    const double df = (double)F[q] - (double)Fref[q];
    sf += df * df;
    phi[q] = (float)(2.0 * wF * df / (3.0 * N_tot));
  }
  red[t] = wE * se / S_tot + wF * sf / (3.0 * N_tot) + wS * ss / (9.0 * S_tot);
  __syncthreads();
  for (int o = 512; o > 0; o >>= 1) {
    if (t < o) red[t] += red[t + o];
    __syncthreads();
  }
  if (t == 0) *loss_part = red[0];
}

// rho(r) = r^2 for |r| <= delta, 2 delta |r| - delta^2 beyond (twice the Huber
// function; delta = inf gives the squared error), and rho'(r).
__device__ __forceinline__ void huber2(double r, double delta, double& rho, double& drho) {
  const double a = fabs(r);
  if (a <= delta) {
    rho = r * r;
    drho = 2.0 * r;
  } else {
    rho = 2.0 * delta * a - delta * delta;
    drho = r < 0.0 ? -2.0 * delta : 2.0 * delta;
  }
}

// Soft threshold of the robust loss: W = exp(-max(z - tau, 0)^2 / 2), dW/dz.
__device__ __forceinline__ void robust_weight(double z, double tau, double& W, double& dW) {
  const double x = z > tau ? z - tau : 0.0;
  W = exp(-0.5 * x * x);
  dW = -x * W;
}

constexpr int kRobustMaxGroups = 256;

// Robust multi-task loss (paper Sec. "Multi-task training strategies"):
//   L = (1/S) sum_s W(z_s, tau)^2 L_s,
//   L_s = w_E rho(E_s/n_s - E_ref,s) + w_F/(3 n_s) sum_{a in s, c} rho(dF_ac) + w_S/9 sum_q rho(dsigma_sq),
//   z_s = (L_s - mu_g) / sd_g over the structures of task g (one group without tasks; z = 0 where sd_g = 0).
// The seeds differentiate the weights too: with A_g = sum W W' L and B_g = sum W W' L z over g,
//   dL/dL_s = (1/S) [W_s^2 + (2/sd_g)(W_s W'_s L_s - A_g/n_g - z_s B_g/n_g)],
// then lam_s, phi_a, Psi_s by the chain rule through L_s.  The statistics couple
// every structure of a task, so the loss runs in three kernels: the base losses
// L_s of each chunk's structures (once its forces and stresses exist), the
// statistics and dL/dL_s over the whole batch, then each chunk's seeds.  Every
// sum runs in a fixed order.

// L_s of the chunk's S structures into Ls[0..S) (one wave per structure: lanes
// over force components, then a fixed butterfly).
__global__ void robust_base_kernel(const double* __restrict__ Ed, const float* __restrict__ Eref,
                                   const int* __restrict__ offsets, int S, const float* __restrict__ F,
                                   const float* __restrict__ Fref, float wE, float wF,
                                   const float* __restrict__ sig, const float* __restrict__ Sref, float wS,
                                   float delta_f, double* __restrict__ Ls) {
  const double delta = (double)delta_f;
  const int lane = threadIdx.x & 63;
  const int nw = (gridDim.x * blockDim.x) >> 6;
  double rho, drho;
  for (int s = (blockIdx.x * blockDim.x + threadIdx.x) >> 6; s < S; s += nw) {
    const int a0 = offsets[s], a1 = offsets[s + 1];
    const double n = (double)(a1 - a0);
    double rf = 0.0;
    for (long long q = 3LL * a0 + lane; q < 3LL * a1; q += 64) {
      huber2((double)F[q] - (double)Fref[q], delta, rho, drho);
      rf += rho;
    }
    rf = wave_sum_d(rf);
    if (lane == 0) {
      huber2(Ed[s] / n - (double)Eref[s], delta, rho, drho);
      double L = wE * rho;
      L += wF * rf / (3.0 * n);
      if (Sref) {
        double rs = 0.0;
        for (int q = 0; q < 9; ++q) {
          huber2((double)sig[9 * s + q] - (double)Sref[9 * s + q], delta, rho, drho);
          rs += rho;
        }
        L += wS * rs / 9.0;
      }
      Ls[s] = L;
    }
  }
}

// Statistics of each task group over the whole batch (structures in order) and
// c_s = dL/dL_s into c[0..S); the loss into *loss.  One workgroup.
__global__ void robust_stats_kernel(const double* __restrict__ Ls, int S, const int* __restrict__ task,
                                    int n_groups, float tau_f, double* __restrict__ c, double* __restrict__ loss) {
  __shared__ double gst[kRobustMaxGroups][6];   // mu, sd, A, B, count, sum W^2 L
  const int t = threadIdx.x;
  const double tau = (double)tau_f;
  for (int g = t; g < n_groups; g += blockDim.x) {
    double cnt = 0.0, sum = 0.0;
    for (int s = 0; s < S; ++s)
      if ((task ? task[s] : 0) == g) {
        cnt += 1.0;
        sum += Ls[s];
      }
    const double mu = cnt > 0.0 ? sum / cnt : 0.0;
    double var = 0.0;
    for (int s = 0; s < S; ++s)
      if ((task ? task[s] : 0) == g) var += (Ls[s] - mu) * (Ls[s] - mu);
    const double sd = cnt > 0.0 ? sqrt(var / cnt) : 0.0;
    double A = 0.0, B = 0.0, lw = 0.0;
    for (int s = 0; s < S; ++s)
      if ((task ? task[s] : 0) == g) {
        const double L = Ls[s];
        const double z = sd > 0.0 ? (L - mu) / sd : 0.0;
        double W, dW;
        robust_weight(z, tau, W, dW);
        A += W * dW * L;
        B += W * dW * L * z;
        lw += W * W * L;
      }
    gst[g][0] = mu; gst[g][1] = sd; gst[g][2] = A; gst[g][3] = B; gst[g][4] = cnt; gst[g][5] = lw;
  }
  __syncthreads();
  for (int s = t; s < S; s += blockDim.x) {
    const int g = task ? task[s] : 0;
    const double L = Ls[s], mu = gst[g][0], sd = gst[g][1];
    const double z = sd > 0.0 ? (L - mu) / sd : 0.0;
    double W, dW;
    robust_weight(z, tau, W, dW);
    double cs = W * W;
    if (sd > 0.0) cs += 2.0 / sd * (W * dW * L - gst[g][2] / gst[g][4] - z * gst[g][3] / gst[g][4]);
    c[s] = cs / (double)S;
  }
  if (t == 0) {
    double lw = 0.0;
    for (int g = 0; g < n_groups; ++g) lw += gst[g][5];
    *loss = lw / (double)S;
  }
}

// Seeds of the chunk's structures and atoms from c = dL/dL_s (c[0..S), the
// chunk's slice): lam_s, Psi_s per structure, phi_a per force component.
__global__ void robust_seed_kernel(const double* __restrict__ Ed, const float* __restrict__ Eref,
                                   const int* __restrict__ offsets, int S, const float* __restrict__ F,
                                   const float* __restrict__ Fref, int N, float wE, float wF,
                                   const float* __restrict__ sig, const float* __restrict__ Sref, float wS,
                                   const float* __restrict__ cell, float delta_f, const double* __restrict__ c,
                                   const int* __restrict__ sid, float* __restrict__ lam, float* __restrict__ phi,
                                   float* __restrict__ Psi) {
  const double delta = (double)delta_f;
  const long long t0 = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  const long long nt = (long long)gridDim.x * blockDim.x;
  double rho, drho;
  for (long long s = t0; s < S; s += nt) {
    const double n = (double)(offsets[s + 1] - offsets[s]);
    huber2(Ed[s] / n - (double)Eref[s], delta, rho, drho);
    lam[s] = (float)(c[s] * wE * drho / n);
    if (Sref) {
      const double iv = 1.0 / cell_volume(cell + 9 * s);
      for (int q = 0; q < 9; ++q) {
        huber2((double)sig[9 * s + q] - (double)Sref[9 * s + q], delta, rho, drho);
        Psi[9 * s + q] = (float)(c[s] * wS / 9.0 * drho * iv);
      }
    }
  }
  for (long long q = t0; q < 3LL * N; q += nt) {
    const int s = sid[q / 3];
    const double n = (double)(offsets[s + 1] - offsets[s]);
    huber2((double)F[q] - (double)Fref[q], delta, rho, drho);
    phi[q] = (float)(c[s] * wF / (3.0 * n) * drho);
  }
}

// loss = sum of the chunk shares in chunk order.
__global__ void loss_total_kernel(const double* __restrict__ part, int n, float* __restrict__ loss) {
  if (threadIdx.x != 0 || blockIdx.x != 0) return;
  double s = 0.0;
  for (int q = 0; q < n; ++q) s += part[q];
  *loss = (float)s;
}

// Chunk-local copies of the neighbour list: atom indices minus a0, edge
// indices minus e0; rowptr of the chunk's atoms and offsets of its structures.
__global__ void rebase_kernel(const int* __restrict__ ei, const int* __restrict__ ej, const int* __restrict__ rev,
                              const int* __restrict__ rowptr, const int* __restrict__ offsets, int a0, int e0, int s0,
                              int n_atoms, long long n_edges, int n_struct, int* __restrict__ cei,
                              int* __restrict__ cej, int* __restrict__ crev, int* __restrict__ crow,
                              int* __restrict__ coff) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q < n_edges) {
    cei[q] = ei[e0 + q] - a0;
    cej[q] = ej[e0 + q] - a0;
    crev[q] = rev[e0 + q] - e0;
  }
  if (q <= n_atoms) crow[q] = rowptr[a0 + q] - e0;
  if (q <= n_struct) coff[q] = offsets[s0 + q] - a0;
}

// First edge of each structure (for the host's chunk plan); indices clamped
// so that offsets that fail validation cannot read out of range.
__global__ void struct_edges_kernel(const int* __restrict__ offsets, const int* __restrict__ rowptr, int S, int N,
                                    int* __restrict__ out) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s > S) return;
  const int a = min(max(offsets[s], 0), N);
  out[s] = rowptr[a];
  out[S + 1 + s] = offsets[s];
}

// rt_e = (phi_i - phi_j) . u_e: the loss adjoint of rbar_e.
// Displacement tangent of the second-order sweep, per edge:
//   gt_e = phi_i - phi_j + Psi_s d_e   (Psi null: no stress term)
//   rt_e = gt_e . u_e
// gt (float4, may be null) is kept for the bond-angle term.
__global__ void rtilde_kernel(const int* __restrict__ ei, const int* __restrict__ ej, const float4* __restrict__ geo,
                              const float* __restrict__ phi, const int* __restrict__ sid,
                              const float* __restrict__ Psi, long long Ne, float* __restrict__ rt,
                              float4* __restrict__ gt) {
  const long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (e >= Ne) return;
  const int i = ei[e], j = ej[e];
  const float4 u = geo[e];
  float gx = phi[3 * i] - phi[3 * j], gy = phi[3 * i + 1] - phi[3 * j + 1], gz = phi[3 * i + 2] - phi[3 * j + 2];
  if (Psi) {
    const float* P = Psi + 9 * sid[i];
    const float dx = u.x * u.w, dy = u.y * u.w, dz = u.z * u.w;
    gx += P[0] * dx + P[1] * dy + P[2] * dz;
    gy += P[3] * dx + P[4] * dy + P[5] * dz;
    gz += P[6] * dx + P[7] * dy + P[8] * dz;
  }
  rt[e] = gx * u.x + gy * u.y + gz * u.z;
  if (gt) gt[e] = make_float4(gx, gy, gz, 0.f);
}

// Readout of the double + final backward, per atom and column:
//   Z   = lam_s SiLU'(z) w_o2 + SiLU''(z) w_o2 vt   (loss adjoint of z)
//   T   = lam_s SiLU(z) + SiLU'(z) vt                (summed over atoms -> dw_o2)
template <int VPL>
__global__ void readout_bwd_kernel(const float* __restrict__ z, const float* __restrict__ vt,
                                   const float* __restrict__ wo2, const float* __restrict__ lam,
                                   const int* __restrict__ sid, int N, int d, float* __restrict__ Z,
                                   float* __restrict__ T) {
  JANUS_WAVE_LOOP(i, N) {
    const float la = lam[sid[i]];
#pragma unroll
    for (int v = 0; v < VPL; ++v) {
      const long long o = i * d + v * 64 + l;
      const float a = z[o], w = wo2[v * 64 + l], q = vt[o];
      const float s = sig(a);
      const float d1 = s + a * s * (1.f - s);
      const float d2 = s * (1.f - s) * (2.f + a * (1.f - 2.f * s));
      Z[o] = la * d1 * w + d2 * w * q;
      T[o] = la * a * s + d1 * q;
    }
  }
}

// Column sums in two fixed-order stages (chunks of 64 rows, then the chunks).
constexpr int kColChunk = 64;
__global__ void colsum_partial_kernel(const float* __restrict__ M, long long rows, int cols,
                                      float* __restrict__ part) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= cols) return;
  const long long r0 = (long long)blockIdx.y * kColChunk, r1 = min(rows, r0 + kColChunk);
  float s = 0.f;
  for (long long r = r0; r < r1; ++r) s += M[r * cols + c];
  part[(long long)blockIdx.y * cols + c] = s;
}
__global__ void colsum_final_kernel(const float* __restrict__ part, int nch, int cols, float* __restrict__ out) {
  const int c = blockIdx.x * blockDim.x + threadIdx.x;
  if (c >= cols) return;
  float s = 0.f;
  for (int q = 0; q < nch; ++q) s += part[(long long)q * cols + c];
  out[c] += s;
}

// Total gate adjoint of (e, c): double-backward part plus the final-backward
// row sums of S~ . SiLU(A) over the column tiles of the slot.
__global__ void gate_total_kernel(const float* __restrict__ g3, const float* __restrict__ gpart,
                                  const int* __restrict__ pos, long long Mk, int ntile, float* __restrict__ gt) {
  const long long f = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (f >= Mk) return;
  float s = g3[f];
  const float* p = gpart + (long long)pos[f] * ntile;
  for (int q = 0; q < ntile; ++q) s += p[q];
  gt[f] = s;
}

// Router logit adjoint of every edge, one thread per (edge, expert x):
//   lt[e, x] = p_e[x] (pt_e[x] - sum_c p_e[eid_ec] gt_ec),  pt_e[x] = sum_c [eid_ec = x] gt_ec,
// with p_e the softmax of the edge's species pair.
__global__ void edge_logit_kernel(const int* __restrict__ pair, const float* __restrict__ pprob,
                                  const int* __restrict__ eid, const float* __restrict__ gt, long long Ne, int k,
                                  int E, float* __restrict__ lt) {
  const long long g = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (g >= Ne * E) return;
  const long long e = g / E;
  const int x = (int)(g - e * E);
  const float* p = pprob + (long long)pair[e] * E;
  float s = 0.f, pt = 0.f;
  for (int c = 0; c < k; ++c) {
    const int y = eid[e * k + c];
    const float gc = gt[e * k + c];
    s += p[y] * gc;
    if (y == x) pt += gc;
  }
  lt[g] = p[x] * (pt - s);
}

// Per atom i and expert x: partC = sum over the edges out of i of lt, partN =
// sum over the edges into i (through rev).  One wave per atom; lane l covers
// expert l % E of the edges l / E, l / E + 64 / E, ... (in order), and the
// 64 / E edge slots of an expert are added in slot order.  E <= 64.
__global__ void router_atom_kernel(const int* __restrict__ rowptr, const int* __restrict__ rev, int E,
                                   const float* __restrict__ lt, int N, float* __restrict__ partC,
                                   float* __restrict__ partN) {
  __shared__ float red[2][256];
  const int slots = kWave / E;
  const int w = threadIdx.x >> 6;
  JANUS_WAVE_LOOP(i, N) {
    const int x = l % E, j = l / E;
    float ac = 0.f, an = 0.f;
    if (j < slots) {
      const int e1 = rowptr[i + 1];
      for (int e = rowptr[i] + j; e < e1; e += slots) {
        ac += lt[(long long)e * E + x];
        an += lt[(long long)rev[e] * E + x];
      }
    }
    red[0][threadIdx.x] = ac;
    red[1][threadIdx.x] = an;
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    if (l < E) {
      float sc = 0.f, sn = 0.f;
      for (int q = 0; q < slots; ++q) {
        sc += red[0][64 * w + q * E + l];
        sn += red[1][64 * w + q * E + l];
      }
      partC[i * E + l] = sc;
      partN[i * E + l] = sn;
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// out[s] += sum over the atoms of species s of rows of M [N, w].  A workgroup
// of 256 threads per species: per pass over min(w, 256) columns, thread t takes
// column t % cols and the atoms g, g + G, ... of the species (g = t / cols,
// G = 256 / cols groups, in atom order); the G group sums of a column are then
// added in group order.
__global__ void species_rows_kernel(const int* __restrict__ sp_off, const int* __restrict__ sp_atoms,
                                    const float* __restrict__ M, int w, int nsp, float* __restrict__ out) {
  __shared__ float red[256];
  const int s = blockIdx.x;
  if (s >= nsp) return;
  const int t = threadIdx.x;
  const int q0 = sp_off[s], q1 = sp_off[s + 1];
  const int cols = w < 256 ? w : 256;
  const int G = 256 / cols;
  const int cl = t % cols, g = t / cols;
  for (int c0 = 0; c0 < w; c0 += cols) {
    const int c = c0 + cl;
    float acc = 0.f;
    if (g < G && c < w)
      for (int q = q0 + g; q < q1; q += G) acc += M[(long long)sp_atoms[q] * w + c];
    red[t] = acc;
    __syncthreads();
    if (g == 0 && c < w) {
      float tot = 0.f;
      for (int j = 0; j < G; ++j) tot += red[j * cols + cl];
      out[(long long)s * w + c] += tot;
    }
    __syncthreads();
  }
}

// Atoms grouped by species in ascending atom order (one wave per species).
__global__ void species_count_kernel(const int* __restrict__ species, int N, int nsp, int* __restrict__ cnt) {
  const int s = blockIdx.x;
  const int l = threadIdx.x;
  int c = 0;
  for (int a0 = 0; a0 < N; a0 += 64) {
    const int a = a0 + l;
    c += __popcll(__ballot(a < N && species[a] == s));
  }
  if (l == 0) cnt[s] = c;
}
__global__ void species_write_kernel(const int* __restrict__ species, int N, const int* __restrict__ sp_off,
                                     int* __restrict__ sp_atoms) {
  const int s = blockIdx.x;
  const int l = threadIdx.x;
  int c = sp_off[s];
  for (int a0 = 0; a0 < N; a0 += 64) {
    const int a = a0 + l;
    const bool m = a < N && species[a] == s;
    const unsigned long long b = __ballot(m);
    if (m) sp_atoms[c + __popcll(b & ((1ull << l) - 1ull))] = a;
    c += __popcll(b);
  }
}

// ------------------------------------------------------------ launch helpers

#define LAUNCH_VPL(kern, d, grid, block, lds, st, ...)                          \
  do {                                                                          \
    switch ((d) / 64) {                                                         \
      case 1: hipLaunchKernelGGL(kern<1>, grid, block, lds, st, __VA_ARGS__); break; \
      case 2: hipLaunchKernelGGL(kern<2>, grid, block, lds, st, __VA_ARGS__); break; \
      case 4: hipLaunchKernelGGL(kern<4>, grid, block, lds, st, __VA_ARGS__); break; \
      case 8: hipLaunchKernelGGL(kern<8>, grid, block, lds, st, __VA_ARGS__); break; \
      default: break;                                                           \
    }                                                                           \
  } while (0)

// Same, for kernels that also take the number of choices per token (1..4).
#define JANUS_LAUNCH_VK_(kern, V, K, grid, block, lds, st, ...) \
  hipLaunchKernelGGL((kern<V, K>), grid, block, lds, st, __VA_ARGS__)
#define JANUS_LAUNCH_K_(kern, V, k, grid, block, lds, st, ...)                           \
  switch (k) {                                                                         \
    case 1: JANUS_LAUNCH_VK_(kern, V, 1, grid, block, lds, st, __VA_ARGS__); break;      \
    case 2: JANUS_LAUNCH_VK_(kern, V, 2, grid, block, lds, st, __VA_ARGS__); break;      \
    case 3: JANUS_LAUNCH_VK_(kern, V, 3, grid, block, lds, st, __VA_ARGS__); break;      \
    case 4: JANUS_LAUNCH_VK_(kern, V, 4, grid, block, lds, st, __VA_ARGS__); break;      \
    default: break;                                                                    \
  }
#define LAUNCH_VPL_K(kern, d, k, grid, block, lds, st, ...)                              \
  do {                                                                                 \
    switch ((d) / 64) {                                                                \
      case 1: JANUS_LAUNCH_K_(kern, 1, k, grid, block, lds, st, __VA_ARGS__); break;     \
      case 2: JANUS_LAUNCH_K_(kern, 2, k, grid, block, lds, st, __VA_ARGS__); break;     \
      case 4: JANUS_LAUNCH_K_(kern, 4, k, grid, block, lds, st, __VA_ARGS__); break;     \
      case 8: JANUS_LAUNCH_K_(kern, 8, k, grid, block, lds, st, __VA_ARGS__); break;     \
      default: break;                                                                  \
    }                                                                                  \
  } while (0)

// Task-aware embedding (paper Sec. "Task-aware feature embedding"), one wave per
// structure s of the chunk:
//   g_s = Tk[task_s] + Qe[charge_s] + Se[spin_s] + (1/n_s) sum_{i in s} Wc[Z_i]
// (the last term is the element fractions times Wc), summed in atom order.
template <int VPL>
__global__ void struct_embed_kernel(const int* __restrict__ task, const int* __restrict__ charge,
                                    const int* __restrict__ spin, const int* __restrict__ offsets,
                                    const int* __restrict__ species, const float* __restrict__ Tk,
                                    const float* __restrict__ Qe, const float* __restrict__ Se,
                                    const float* __restrict__ Wc, int S, int d, float* __restrict__ g) {
  JANUS_WAVE_LOOP(s, S) {
    float c[VPL], acc[VPL];
    zero_row<VPL>(c);
    const int a0 = offsets[s], a1 = offsets[s + 1];
    for (int i = a0; i < a1; ++i) {
      float w[VPL];
      ld_row<VPL>(Wc + (long long)species[i] * d, l, w);
      add_row<VPL>(c, w);
    }
    const float inv = a1 > a0 ? 1.f / (float)(a1 - a0) : 0.f;
    ld_row<VPL>(Tk + (long long)task[s] * d, l, acc);
    float w[VPL];
    ld_row<VPL>(Qe + (long long)charge[s] * d, l, w);
    add_row<VPL>(acc, w);
    ld_row<VPL>(Se + (long long)spin[s] * d, l, w);
    add_row<VPL>(acc, w);
#pragma unroll
    for (int v = 0; v < VPL; ++v) acc[v] += c[v] * inv;
    st_row<VPL>(g + s * d, l, acc);
  }
}

// h0_i += g_s(i)
__global__ void add_struct_rows_kernel(const float* __restrict__ g, const int* __restrict__ sid, int N, int d,
                                       float* __restrict__ h) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (long long)N * d) return;
  const long long i = q / d;
  h[q] += g[(long long)sid[i] * d + (q - i * d)];
}

// gbar_s = sum over the atoms of s (in order) of hbar_i, one wave per structure.
template <int VPL>
__global__ void struct_sum_kernel(const int* __restrict__ offsets, const float* __restrict__ hbar, int S, int d,
                                  float* __restrict__ gbar) {
  JANUS_WAVE_LOOP(s, S) {
    float acc[VPL];
    zero_row<VPL>(acc);
    for (int i = offsets[s]; i < offsets[s + 1]; ++i) {
      float x[VPL];
      ld_row<VPL>(hbar + (long long)i * d, l, x);
      add_row<VPL>(acc, x);
    }
    st_row<VPL>(gbar + s * d, l, acc);
  }
}

// out[t] += sum over the structures s with label[s] == t (in order) of gbar_s;
// one workgroup per label value.
__global__ void label_rows_kernel(const int* __restrict__ label, int S, const float* __restrict__ gbar, int d,
                                  float* __restrict__ out) {
  const int t = blockIdx.x;
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float acc = 0.f;
    for (int s = 0; s < S; ++s)
      if (label[s] == t) acc += gbar[(long long)s * d + c];
    out[(long long)t * d + c] += acc;
  }
}

// dWc[z] += sum over the atoms i of species z (in atom order) of gbar_s(i) / n_s(i).
__global__ void comp_rows_kernel(const int* __restrict__ sp_off, const int* __restrict__ sp_atoms,
                                 const int* __restrict__ sid, const int* __restrict__ offsets,
                                 const float* __restrict__ gbar, int d, int nsp, float* __restrict__ out) {
  const int z = blockIdx.x;
  if (z >= nsp) return;
  for (int c = threadIdx.x; c < d; c += blockDim.x) {
    float acc = 0.f;
    for (int q = sp_off[z]; q < sp_off[z + 1]; ++q) {
      const int i = sp_atoms[q], s = sid[i];
      acc += gbar[(long long)s * d + c] / (float)(offsets[s + 1] - offsets[s]);
    }
    out[(long long)z * d + c] += acc;
  }
}

// flag[0] = 1 when a structure's label is out of its table's range.
__global__ void validate_labels_kernel(const int* __restrict__ task, const int* __restrict__ charge,
                                       const int* __restrict__ spin, int S, int nt, int nc, int ns,
                                       int* __restrict__ flag) {
  const int s = blockIdx.x * blockDim.x + threadIdx.x;
  if (s >= S) return;
  if (task[s] < 0 || task[s] >= nt || charge[s] < 0 || charge[s] >= nc || spin[s] < 0 || spin[s] >= ns)
    atomicOr(flag, 1);
}

// h0_i = A[Z_i]
__global__ void species_rows_gather_kernel(const float* __restrict__ A, const int* __restrict__ species, int N, int d,
                                           float* __restrict__ h) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q >= (long long)N * d) return;
  const long long i = q / d;
  h[q] = A[(long long)species[i] * d + (q - i * d)];
}

// Workgroups of four waves over `items`, at most 2048: one full set of resident
// workgroups (256 CUs x 8 of them at 8 waves per SIMD), each wave then looping over
// its items.  The edge kernels stage W_b in LDS once per workgroup; with 8192
// workgroups they ran 13-16 % longer on the small batch (4096 and 1024: 5 % and
// 30 % longer than 2048).
inline dim3 wave_grid(long long items) {
  long long blocks = (items + 3) / 4;
  if (blocks > 2048) blocks = 2048;
  if (blocks < 1) blocks = 1;
  return dim3((unsigned)blocks);
}

// ------------------------------------------------------------ weight layout

struct Layout {
  struct Ent {
    std::string name;
    long long off;
    int ndim;
    long long shape[3];
  };
  std::vector<Ent> ents;
  long long total = 0;
  void add(const std::string& n, std::initializer_list<long long> sh) {
    Ent e;
    e.name = n;
    e.off = total;
    e.ndim = (int)sh.size();
    long long sz = 1;
    int q = 0;
    for (long long s : sh) {
      e.shape[q++] = s;
      sz *= s;
    }
    for (; q < 3; ++q) e.shape[q] = 0;
    ents.push_back(e);
    total += sz;
  }
  long long at(const std::string& n) const {
    for (const auto& e : ents)
      if (e.name == n) return e.off;
    return -1;
  }
};

Layout make_layout(const janus_config& c) {
  Layout L;
  const long long S = c.n_species, d = c.d, E = c.n_experts, h = c.d_hidden, nb = c.n_rbf;
  L.add("A", {S, d});
  if (c.n_tasks) {
    L.add("Tk", {(long long)c.n_tasks, d});
    L.add("Qe", {(long long)c.n_charges, d});
    L.add("Se", {(long long)c.n_spins, d});
    L.add("Wc", {S, d});
  }
  for (int t = 0; t < c.n_blocks; ++t) {
    const std::string p = "blocks." + std::to_string(t) + ".";
    L.add(p + "W_b", {nb, d});
    L.add(p + "Pc", {S, E});
    L.add(p + "Pn", {S, E});
    L.add(p + "beta", {E});
    if (c.route_feat) L.add(p + "Wr", {d, E});
    L.add(p + "W1", {E, d, h});
    L.add(p + "W2", {E, h, d});
    if (c.three_body) {
      const long long E3 = c.n_experts3, h3 = c.d_hidden3, nf = (long long)c.n_legendre * nb;
      L.add(p + "W_a", {nf, d});
      L.add(p + "P3a", {S, E3});
      L.add(p + "P3b", {S, E3});
      L.add(p + "P3c", {S, E3});
      L.add(p + "beta3", {E3});
      L.add(p + "W1a", {E3, d, h3});
      L.add(p + "W2a", {E3, h3, d});
    }
    if (c.atom_moe) {
      const long long Ef = c.n_experts_f, hf = c.d_hidden_f;
      L.add(p + "Pf", {S, Ef});
      L.add(p + "betaf", {Ef});
      L.add(p + "W1f", {Ef, d, hf});
      L.add(p + "W2f", {Ef, hf, d});
    }
    if (c.n_heads) {
      L.add(p + "Wqkv", {d, 3 * d});
      L.add(p + "Wo", {d, d});
    }
  }
  L.add("W_o1", {d, d});
  L.add("w_o2", {d});
  return L;
}

int check_config(const janus_config* c) {
  if (!c) return JANUS_EINVAL;
  if (c->n_species < 1 || c->n_species > 128 || c->d < 64 || c->n_rbf < 1 || c->n_rbf > 32 || c->n_blocks < 0 ||
      c->n_blocks > 16 || c->n_experts < 1 || c->n_experts > 64 || c->top_k < 1 || c->top_k > 4 ||
      c->top_k > c->n_experts || c->d_hidden < 64 || !(c->r_cut > 0.f))
    return JANUS_EINVAL;
  if (c->d % 64 || (c->d / 64 != 1 && c->d / 64 != 2 && c->d / 64 != 4 && c->d / 64 != 8) || c->d_hidden % 64 ||
      c->n_rbf % 4 || c->env_p != 6)
    return JANUS_EUNSUPPORTED;
  if (c->three_body) {
    if (c->n_experts3 < 1 || c->n_experts3 > 64 || c->top_k3 < 1 || c->top_k3 > 4 || c->top_k3 > c->n_experts3 ||
        c->d_hidden3 < 64 || c->n_legendre < 1 || !(c->r_cut3 > 0.f) || c->r_cut3 > c->r_cut)
      return JANUS_EINVAL;
    // the feature-to-width matrix W_a is staged in LDS (at most 64 KB)
    if (c->d_hidden3 % 64 || c->n_legendre > 8 || (size_t)c->n_legendre * c->n_rbf * c->d * 4 > 65536)
      return JANUS_EUNSUPPORTED;
  }
  if (!(c->w_S >= 0.f)) return JANUS_EINVAL;
  if (c->n_heads < 0 || (c->n_heads && c->d % c->n_heads)) return JANUS_EINVAL;
  if (c->n_tasks < 0 || (c->n_tasks && (c->n_charges < 1 || c->n_spins < 1))) return JANUS_EINVAL;
  if (c->robust != 0 && c->robust != 1) return JANUS_EINVAL;
  if (c->robust && (!(c->huber_delta > 0.f) || c->robust_tau != c->robust_tau)) return JANUS_EINVAL;
  if (c->robust && c->n_tasks > kRobustMaxGroups) return JANUS_EUNSUPPORTED;

  // heads of 32, 64 or 128 columns
  if (c->n_heads && c->d / c->n_heads != 32 && c->d / c->n_heads != 64 && c->d / c->n_heads != 128)
    return JANUS_EUNSUPPORTED;
  if (c->route_feat != 0 && c->route_feat != 1) return JANUS_EINVAL;
  if (c->atom_moe) {
    if (c->n_experts_f < 1 || c->n_experts_f > 64 || c->top_k_f < 1 || c->top_k_f > 4 ||
        c->top_k_f > c->n_experts_f || c->d_hidden_f < 64)
      return JANUS_EINVAL;
    if (c->d_hidden_f % 64) return JANUS_EUNSUPPORTED;
  }
  return JANUS_OK;
}

// ------------------------------------------------------------ workspace plan

struct Plan {
  // shared
  int* flag;
  int* sid;
  float4* geo;
  float *B, *dB, *rt, *rbar;
  float *d2B, *rpos;   // loss gradient in positions: B''(r_e) and dL/dr_e (null without it)
  int *sp_cnt, *sp_off, *sp_atoms;
  float *z, *eps, *lam, *phi, *vt, *Zr, *Tr, *colpart, *sig, *Psi, *gs, *gsb;
  float4* gtan;
  double* Ed;
  float *h, *hh, *hht, *h3;   // [(T+1) or T][N, d]; the final-backward adjoint reuses hh
  // routing, per block
  int *peid, *pair, *eid, *pos, *total, *off, *cnt, *colpre;
  float *pgate, *pprob, *gate, *slot_gate;
  RowsTile* tiles;
  int* ntiles;
  WChunk* chunks;
  int *nchunks, *cfirst;
  // dense tables: atoms (group of N rows) and edges (group of Ne rows)
  int *rowN, *rowE;
  RowsTile* tilesN;
  int* ntN;
  WChunk *chunksN, *chunksE;
  int *ncN, *cfN, *ncE, *cfE;
  // per block activations
  float *Xs, *A, *Sb, *Ab, *Ybs, *Xbar, *Fbar, *g3;
  // temporaries
  float *T1, *T2, *Pe, *Ft, *gpart, *gt, *partC, *partN, *lte, *partial;
  // expert weight-gradient partials (the side stream's own) and the double
  // backward's Sbt of block 0 (block t > 0 writes it over Abar of block t-1)
  float *partial2, *Shat0;
  // chunk-local neighbour list (indices relative to the chunk)
  int *cei, *cej, *crev, *crow, *coff;
  long long* scan;   // scratch of the exclusive scans (triplet CSR, species groups)
  // three-body term: triplets (CSR by first edge), per-edge basis at r3,
  // per-block triplet routing, activations and adjoints
  int *tcount, *trow, *te, *te2, *trev;
  float *tc, *B3, *dB3, *u3, *du3;
  float4 *tacc, *tct, *gvec;
  float4* tlane;   // per-triplet scalars in second-edge order (tri_lane_kernel)
  int *eid3, *pos3, *total3, *off3, *cnt3, *colpre3;
  int* pos3r;      // pos3 in second-edge order, per block
  float *gate3, *slot_gate3, *g3t;
  RowsTile* tiles3;
  int* ntiles3;
  WChunk* chunks3;
  int *nchunks3, *cfirst3;
  int *rowT;
  WChunk* chunksT;
  int *ncT, *cfT;
  // loss gradient in positions with the bond-angle term: row tiles over the
  // triplets, feature adjoints of the final and double backward [Nt, nf],
  // per-triplet and per-edge displacement vectors (null without it)
  RowsTile* tilesT;
  int* ntT;
  int mtT;
  float *adjG, *adjGd;
  float4 *tp1, *tp2, *tpos;
  float *Z3s, *A3, *S3b, *A3b, *Y3bs, *Zbar3;
  float *Q, *LT3, *VT, *G3f, *G3t, *T3a, *T3b, *gpart3, *gt3, *LB, *LC, *pa, *pb, *pc;
  // feature-update MoE: atom tokens (one row per atom in an identity CSR),
  // per-block routing by species, GEMM tables, activations and adjoints
  int* iota;
  int *seid, *eidf, *posf, *totalf, *offf, *cntf, *colpref;
  float *sgate, *sprob, *gatef, *slot_gatef, *g3f;
  RowsTile* tilesf;
  int* ntilesf;
  WChunk* chunksf;
  int *nchunksf, *cfirstf;
  float *Xsf, *Af, *Sbf, *Abf, *Ybf, *uu, *T1f, *T2f, *ut, *gpartf, *gtf, *ltf;
  // neighbourhood attention: per block messages, q|k|v, softmax statistics, atom
  // sums, first-order adjoints, tangents; temporaries; GEMM tables over Ne rows
  float *eu, *eud;
  float *Mm, *QKV, *stats, *osum, *OB, *QKVb, *MB, *Mh, *QKVh;
  float *AO, *QKVa, *mta, *osh, *rbh;
  float *rbs, *rlh;   // with the loss gradient in positions: dE/du per block and edge, log-u adjoints
  RowsTile* tilesE;
  int* ntE;
  WChunk* chunksA;
  int *ncA, *cfA;
  // sizes
  int T, E, k, d, hdim, nb, nsp, N, S;
  long long Ne, M;
  int mt, mc, kc, mtN, kcN, mcN, kcE, mcE, nch, ntile;
  int three, E3, k3, hd3, L3, nf;
  long long Nt, M3;
  int mt3, mc3, kc3, kcT, mcT, nch3, ntile3;
  int atom, Ef, kf, hdf;
  long long Mf;
  int mtf, kcf, mcf, nchf, ntilef;
  int attn, H, mtE, kcA, mcA;
  // routing on the edge tokens: per block the edge tokens [Ne, d], the expert outputs
  // before gating [M, d], the full softmax [Ne, Ep], the phase-2 gate and logit
  // adjoints, the phase-3 gate adjoints and softmax adjoints, the padded router
  // weight and its gradient [d, Ep]; temporaries over the edges; the phase-2 atom
  // adjoints kept for phase 4; a row of ones (gates already applied); the weight
  // gradient's chunk table over the edges
  int rf, Ep, kcR, mcR;
  float *Xe, *Yst, *fprob, *gbar, *lbar, *P3, *gh, *WrP, *dWrP, *Lw, *Xadd, *Xh, *hh2, *ones, *wrpart;
  int *iotaE, *ncR, *cfR;
  WChunk* chunksR;
};

size_t plan_layout(Plan& p, void* base, const janus_config& c, int N, int S, long long Ne, long long Nt = 0,
                   bool pos_grad = false) {
  Carver cv(base);
  p.T = c.n_blocks;
  p.E = c.n_experts;
  p.k = c.top_k;
  p.d = c.d;
  p.hdim = c.d_hidden;
  p.nb = c.n_rbf;
  p.nsp = c.n_species;
  p.N = N;
  p.S = S;
  p.Ne = Ne;
  p.M = Ne * c.top_k;
  const int T = p.T, E = p.E, d = p.d, h = p.hdim;
  const long long M = p.M, Nd = (long long)N * d;
  const long long np = (long long)p.nsp * p.nsp;
  p.mt = max_rows_tiles(M, E);
  p.kc = wgrad_chunk_rows(M, d, h);
  p.mc = max_wchunks(M, E, p.kc);
  p.mtN = max_rows_tiles(N, 1);
  p.kcN = wgrad_chunk_rows(N, d, d);
  p.mcN = max_wchunks(N, 1, p.kcN);
  p.kcE = skinny_chunk_rows(Ne, p.nb, d);
  p.mcE = max_wchunks(Ne, 1, p.kcE);
  p.nch = sort_chunks(M);
  p.ntile = (h + GBN - 1) / GBN;

  p.flag = cv.take<int>(4);
  p.sid = cv.take<int>(N);
  p.geo = cv.take<float4>(Ne);
  p.B = cv.take<float>(Ne * p.nb);
  p.dB = cv.take<float>(Ne * p.nb);
  p.rt = cv.take<float>(Ne);
  p.rbar = cv.take<float>(Ne);
  p.d2B = pos_grad ? cv.take<float>(Ne * p.nb) : nullptr;
  p.rpos = pos_grad ? cv.take<float>(Ne + 1) : nullptr;
  p.sp_cnt = cv.take<int>(p.nsp);
  p.scan = cv.take<long long>(scan_scratch_bytes(std::max<long long>(Ne, p.nsp)) / sizeof(long long));
  p.sp_off = cv.take<int>(p.nsp + 1);
  p.sp_atoms = cv.take<int>(N);
  p.z = cv.take<float>(Nd);
  p.eps = cv.take<float>(N);
  p.lam = cv.take<float>(S);
  p.phi = cv.take<float>(3LL * N);
  p.sig = cv.take<float>(9LL * S);
  p.gs = cv.take<float>((long long)S * d + 4);
  p.gsb = cv.take<float>((long long)S * d + 4);
  p.Psi = cv.take<float>(9LL * S);
  p.gtan = cv.take<float4>(Ne + 1);
  p.vt = cv.take<float>(Nd);
  p.Zr = cv.take<float>(Nd);
  p.Tr = cv.take<float>(Nd);
  p.colpart = cv.take<float>(((N + kColChunk - 1) / kColChunk) * (long long)d);
  p.Ed = cv.take<double>(S);
  p.h = cv.take<float>((T + 1) * Nd);
  p.hh = cv.take<float>((T + 1) * Nd);
  p.hht = cv.take<float>((T + 1) * Nd);
  p.h3 = cv.take<float>(T * Nd + 1);

  p.peid = cv.take<int>(T * np * p.k);
  p.pgate = cv.take<float>(T * np * p.k);
  p.pprob = cv.take<float>(T * np * E);
  p.pair = cv.take<int>(T * Ne);
  p.eid = cv.take<int>(T * M);
  p.gate = cv.take<float>(T * M);
  p.pos = cv.take<int>(T * M);
  p.slot_gate = cv.take<float>(T * M);
  p.total = cv.take<int>(T * E);
  p.off = cv.take<int>(T * (E + 1));
  p.cnt = cv.take<int>((long long)p.nch * E + 1);
  p.colpre = cv.take<int>((long long)p.nch * E + 1);
  p.tiles = cv.take<RowsTile>((long long)T * p.mt);
  p.ntiles = cv.take<int>(T + 1);
  p.chunks = cv.take<WChunk>((long long)T * p.mc);
  p.nchunks = cv.take<int>(T + 1);
  p.cfirst = cv.take<int>(T * (E + 1) + 1);

  p.rowN = cv.take<int>(2);
  p.rowE = cv.take<int>(2);
  p.tilesN = cv.take<RowsTile>(p.mtN);
  p.ntN = cv.take<int>(1);
  p.chunksN = cv.take<WChunk>(p.mcN);
  p.ncN = cv.take<int>(1);
  p.cfN = cv.take<int>(2);
  p.chunksE = cv.take<WChunk>(p.mcE);
  p.ncE = cv.take<int>(1);
  p.cfE = cv.take<int>(2);

  p.Xs = cv.take<float>(T * M * d);
  p.A = cv.take<float>(T * M * h);
  p.Sb = cv.take<float>(T * M * h);
  p.Ab = cv.take<float>(T * M * h);
  p.Ybs = cv.take<float>(T * M * d);
  p.Xbar = cv.take<float>(T * Ne * d);
  p.Fbar = cv.take<float>(T * Ne * d);
  p.g3 = cv.take<float>(T * M);

  p.T1 = cv.take<float>(M * d);
  p.T2 = cv.take<float>(M * d);
  p.Pe = cv.take<float>(Ne * d);
  p.Ft = cv.take<float>(Ne * d);
  p.gpart = cv.take<float>(M * p.ntile);
  p.gt = cv.take<float>(M);
  p.partC = cv.take<float>((long long)N * E);
  p.partN = cv.take<float>((long long)N * E);
  p.lte = cv.take<float>(Ne * E + 1);
  long long part = (long long)p.mc * d * h;
  part = std::max(part, (long long)p.mcN * d * d);
  part = std::max(part, (long long)p.mcE * p.nb * d);
  if (c.three_body) {   // triplet expert and W_a gradients (same chunking as below)
    const long long M3 = Nt * c.top_k3;
    const int nf = c.n_legendre * c.n_rbf;
    part = std::max(part, (long long)max_wchunks(M3, c.n_experts3, wgrad_chunk_rows(M3, d, c.d_hidden3)) * d *
                              c.d_hidden3);
    part = std::max(part, (long long)max_wchunks(Nt, 1, wgrad_chunk_rows(Nt, nf, d)) * nf * d);
  }
  p.atom = c.atom_moe ? 1 : 0;
  p.Ef = c.n_experts_f;
  p.kf = c.top_k_f;
  p.hdf = c.d_hidden_f;
  p.Mf = p.atom ? (long long)N * c.top_k_f : 0;
  if (p.atom) {
    p.mtf = max_rows_tiles(p.Mf, p.Ef);
    p.kcf = wgrad_chunk_rows(p.Mf, d, p.hdf);
    p.mcf = max_wchunks(p.Mf, p.Ef, p.kcf);
    p.nchf = sort_chunks(p.Mf);
    p.ntilef = (p.hdf + GBN - 1) / GBN;
    part = std::max(part, (long long)p.mcf * d * p.hdf);
  }
  p.attn = c.n_heads ? 1 : 0;
  p.H = c.n_heads;
  p.rf = c.route_feat ? 1 : 0;
  p.Ep = (E + 15) / 16 * 16;
  p.mtE = max_rows_tiles(Ne, 1);
  if (p.rf) {
    p.kcR = wgrad_chunk_rows(Ne, d, p.Ep);
    p.mcR = max_wchunks(Ne, 1, p.kcR);
  }
  if (p.attn) {
    p.kcA = wgrad_chunk_rows(Ne, d, 3 * d);
    p.mcA = max_wchunks(Ne, 1, p.kcA);
    part = std::max(part, (long long)p.mcA * d * 3 * d);
  }
  p.partial = cv.take<float>(part);
  p.partial2 = cv.take<float>((long long)p.mc * d * h);
  p.Shat0 = cv.take<float>(M * h);
  p.cei = cv.take<int>(Ne + 1);
  p.cej = cv.take<int>(Ne + 1);
  p.crev = cv.take<int>(Ne + 1);
  p.crow = cv.take<int>(N + 1);
  p.coff = cv.take<int>(S + 1);

  p.three = c.three_body ? 1 : 0;
  p.Nt = p.three ? Nt : 0;
  p.E3 = c.n_experts3;
  p.k3 = c.top_k3;
  p.hd3 = c.d_hidden3;
  p.L3 = c.n_legendre;
  p.nf = c.n_legendre * c.n_rbf;
  p.M3 = p.Nt * c.top_k3;
  p.tilesT = nullptr;
  p.ntT = nullptr;
  p.adjG = p.adjGd = nullptr;
  p.tp1 = p.tp2 = p.tpos = nullptr;
  if (p.three) {
    const long long M3 = p.M3, Ntt = p.Nt, h3 = p.hd3, E3 = p.E3;
    p.mt3 = max_rows_tiles(M3, p.E3);
    p.kc3 = wgrad_chunk_rows(M3, d, p.hd3);
    p.mc3 = max_wchunks(M3, p.E3, p.kc3);
    p.kcT = wgrad_chunk_rows(Ntt, p.nf, d);
    p.mcT = max_wchunks(Ntt, 1, p.kcT);
    p.nch3 = sort_chunks(M3);
    p.ntile3 = (p.hd3 + GBN - 1) / GBN;
    p.tcount = cv.take<int>(Ne + 1);
    p.trow = cv.take<int>(Ne + 1);
    p.te = cv.take<int>(Ntt + 1);
    p.te2 = cv.take<int>(Ntt + 1);
    p.trev = cv.take<int>(Ntt + 1);
    p.tc = cv.take<float>(Ntt + 1);
    p.B3 = cv.take<float>(Ne * p.nb + 4);
    p.dB3 = cv.take<float>(Ne * p.nb + 4);
    p.u3 = cv.take<float>(Ne + 1);
    p.du3 = cv.take<float>(Ne + 1);
    p.tacc = cv.take<float4>(Ntt + 1);
    p.tct = cv.take<float4>(Ntt + 1);
    p.gvec = cv.take<float4>(Ne + 1);
    p.tlane = cv.take<float4>(Ntt + 1);
    p.eid3 = cv.take<int>(T * M3 + 1);
    p.gate3 = cv.take<float>(T * M3 + 1);
    p.pos3 = cv.take<int>(T * M3 + 1);
    p.pos3r = cv.take<int>(T * M3 + 1);
    p.slot_gate3 = cv.take<float>(T * M3 + 1);
    p.g3t = cv.take<float>(T * M3 + 1);
    p.total3 = cv.take<int>(T * E3);
    p.off3 = cv.take<int>(T * (E3 + 1));
    p.cnt3 = cv.take<int>((long long)p.nch3 * E3 + 1);
    p.colpre3 = cv.take<int>((long long)p.nch3 * E3 + 1);
    p.tiles3 = cv.take<RowsTile>((long long)T * p.mt3);
    p.ntiles3 = cv.take<int>(T + 1);
    p.chunks3 = cv.take<WChunk>((long long)T * p.mc3);
    p.nchunks3 = cv.take<int>(T + 1);
    p.cfirst3 = cv.take<int>(T * (E3 + 1) + 1);
    p.rowT = cv.take<int>(2);
    p.chunksT = cv.take<WChunk>(p.mcT);
    p.mtT = max_rows_tiles(Ntt, 1);
    p.tilesT = pos_grad ? cv.take<RowsTile>(p.mtT) : nullptr;
    p.ntT = pos_grad ? cv.take<int>(1) : nullptr;
    p.adjG = pos_grad ? cv.take<float>(Ntt * p.nf + 4) : nullptr;
    p.adjGd = pos_grad ? cv.take<float>(Ntt * p.nf + 4) : nullptr;
    p.tp1 = pos_grad ? cv.take<float4>(Ntt + 1) : nullptr;
    p.tp2 = pos_grad ? cv.take<float4>(Ntt + 1) : nullptr;
    p.tpos = pos_grad ? cv.take<float4>(Ne + 1) : nullptr;
    p.ncT = cv.take<int>(1);
    p.cfT = cv.take<int>(2);
    p.Z3s = cv.take<float>(T * M3 * d + 4);
    p.A3 = cv.take<float>(T * M3 * h3 + 4);
    p.S3b = cv.take<float>(T * M3 * h3 + 4);
    p.A3b = cv.take<float>(T * M3 * h3 + 4);
    p.Y3bs = cv.take<float>(T * M3 * d + 4);
    p.Zbar3 = cv.take<float>(T * Ntt * d + 4);
    p.Q = cv.take<float>(Ne * d + 4);
    p.LT3 = cv.take<float>(Ntt * E3 + 4);
    p.VT = cv.take<float>(Ntt * d + 4);
    p.G3f = cv.take<float>(Ntt * p.nf + 4);
    p.G3t = cv.take<float>(Ntt * p.nf + 4);
    p.T3a = cv.take<float>(M3 * d + 4);
    p.T3b = cv.take<float>(M3 * d + 4);
    p.gpart3 = cv.take<float>(M3 * p.ntile3 + 4);
    p.gt3 = cv.take<float>(M3 + 1);
    p.LB = cv.take<float>(Ne * E3 + 1);
    p.LC = cv.take<float>(Ne * E3 + 1);
    p.pa = cv.take<float>((long long)N * E3 + 1);
    p.pb = cv.take<float>((long long)N * E3 + 1);
    p.pc = cv.take<float>((long long)N * E3 + 1);
  }
  if (p.atom) {
    const long long Mf = p.Mf, Ef = p.Ef, kf = p.kf, hf = p.hdf;
    p.iota = cv.take<int>(N + 1);
    p.seid = cv.take<int>(T * p.nsp * kf);
    p.sgate = cv.take<float>(T * p.nsp * kf);
    p.sprob = cv.take<float>(T * p.nsp * Ef);
    p.eidf = cv.take<int>(T * Mf + 1);
    p.gatef = cv.take<float>(T * Mf + 1);
    p.posf = cv.take<int>(T * Mf + 1);
    p.slot_gatef = cv.take<float>(T * Mf + 1);
    p.g3f = cv.take<float>(T * Mf + 1);
    p.totalf = cv.take<int>(T * Ef);
    p.offf = cv.take<int>(T * (Ef + 1));
    p.cntf = cv.take<int>((long long)p.nchf * Ef + 1);
    p.colpref = cv.take<int>((long long)p.nchf * Ef + 1);
    p.tilesf = cv.take<RowsTile>((long long)T * p.mtf);
    p.ntilesf = cv.take<int>(T + 1);
    p.chunksf = cv.take<WChunk>((long long)T * p.mcf);
    p.nchunksf = cv.take<int>(T + 1);
    p.cfirstf = cv.take<int>(T * (Ef + 1) + 1);
    p.Xsf = cv.take<float>(T * Mf * d + 4);
    p.Af = cv.take<float>(T * Mf * hf + 4);
    p.Sbf = cv.take<float>(T * Mf * hf + 4);
    p.Abf = cv.take<float>(T * Mf * hf + 4);
    p.Ybf = cv.take<float>(T * Mf * d + 4);
    p.uu = cv.take<float>(T * Nd + 4);
    p.T1f = cv.take<float>(Mf * d + 4);
    p.T2f = cv.take<float>(Mf * d + 4);
    p.ut = cv.take<float>(Nd + 4);
    p.gpartf = cv.take<float>(Mf * p.ntilef + 4);
    p.gtf = cv.take<float>(Mf + 1);
    p.ltf = cv.take<float>((long long)N * Ef + 1);
  }
  p.rbs = p.rlh = nullptr;
  if (p.attn) {
    const long long Ed = Ne * d + 4, E3d = 3 * Ne * d + 4;
    p.eu = cv.take<float>(Ne + 1);
    p.eud = cv.take<float>(Ne + 1);
    p.Mm = cv.take<float>(T * Ed);
    p.QKV = cv.take<float>(T * E3d);
    p.stats = cv.take<float>(T * (2 * Ne * p.H + 4));
    p.osum = cv.take<float>(T * Nd + 4);
    p.OB = cv.take<float>(T * Nd + 4);
    p.QKVb = cv.take<float>(T * E3d);
    p.MB = cv.take<float>(T * Ed);
    p.Mh = cv.take<float>(T * Ed);
    p.QKVh = cv.take<float>(T * E3d);
    p.AO = cv.take<float>(Nd + 4);
    p.QKVa = cv.take<float>(E3d);
    p.mta = cv.take<float>(Ed);
    p.osh = cv.take<float>(Nd + 4);
    p.rbh = cv.take<float>(Ne * p.H + 4);
    p.rbs = pos_grad ? cv.take<float>((long long)T * Ne + 4) : nullptr;
    p.rlh = pos_grad ? cv.take<float>(Ne * p.H + 4) : nullptr;
    p.chunksA = cv.take<WChunk>(p.mcA);
    p.ncA = cv.take<int>(1);
    p.cfA = cv.take<int>(2);
  }
  p.tilesE = nullptr;
  p.ntE = nullptr;
  if (p.attn || p.rf) {
    p.tilesE = cv.take<RowsTile>(p.mtE);
    p.ntE = cv.take<int>(1);
  }
  if (p.rf) {
    const long long Ep = p.Ep, Ed = Ne * d + 4;
    p.Xe = cv.take<float>(T * Ed);
    p.Yst = cv.take<float>(T * (M * d + 4));
    p.fprob = cv.take<float>(T * (Ne * Ep + 4));
    p.gbar = cv.take<float>(T * M + 4);
    p.lbar = cv.take<float>(T * (Ne * Ep + 4));
    p.P3 = cv.take<float>(T * (Ne * Ep + 4));
    p.gh = cv.take<float>(T * M + 4);
    p.WrP = cv.take<float>(T * d * Ep);
    p.dWrP = cv.take<float>(T * d * Ep);
    p.Lw = cv.take<float>(Ne * Ep + 4);
    p.Xadd = cv.take<float>(Ed);
    p.Xh = cv.take<float>(Ed);
    p.hh2 = cv.take<float>((T + 1) * Nd + 4);
    p.ones = cv.take<float>(M + 4);
    p.wrpart = cv.take<float>((long long)p.mcR * d * Ep + 4);
    p.iotaE = cv.take<int>(Ne + 1);
    p.chunksR = cv.take<WChunk>(p.mcR);
    p.ncR = cv.take<int>(1);
    p.cfR = cv.take<int>(2);
  }
  return cv.size();
}

__global__ void fill_kernel(float* __restrict__ out, long long n, float v) {
  const long long q = (long long)blockIdx.x * blockDim.x + threadIdx.x;
  if (q < n) out[q] = v;
}

// Identity CSR [0, 1, ..., N]: every atom is one token of the feature-update MoE.
__global__ void iota_kernel(int* __restrict__ out, int n) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q <= n) out[q] = q;
}

__global__ void set_rows_kernel(int* rowN, int N, int* rowE, long long Ne) {
  if (threadIdx.x == 0) {
    rowN[0] = 0;
    rowN[1] = N;
    rowE[0] = 0;
    rowE[1] = (int)Ne;
  }
}

}  // namespace janus

